// split_impl.h -- internal interface of split evaluation and partitioning
// (split.hip) used by the tree driver.
#pragma once

#include "common.h"

namespace gbt {

struct EvalParams {
    double lambda;
    double gamma;
    double mcw;
    int32_t e_g;
    int32_t e_h;
    const int32_t *e_dev;  // when set, {e_g, e_h} are read from device memory
};

struct EvalNode {
    long long sum_g, sum_h;
    int32_t slot;   // histogram slot
    int32_t heap;   // node id
};

struct EvalCand {
    double gain;
    long long lg, lh;
    int32_t feature;
    int32_t split_bin;
    int32_t default_left;
    int32_t valid;
};

// n_nodes sizes the grid; when n_nodes_d is given the live count is read
// from device memory (at most n_nodes).
gbt_status eval_impl(gbt_ctx *c, const gbt_matrix *mx, const int64_t *hist, const EvalNode *nodes_d,
                     int32_t n_nodes, const EvalParams &ep, gbt_split *out_d,
                     const int32_t *n_nodes_d = nullptr, DevNode *decide = nullptr);
// Stable partition of rows[0, n) by each slot's node (slot_node[i], or
// position[rows[i]] when slot_node is NULL): the rows of every splitting
// node go left or right within its segment.  rows_out receives the new
// order, slot_node_out (if not NULL) each new slot's node; when
// slot_node_out is NULL, position[row] receives the child of every row of a
// splitting node.  nodes[id].pleft / nleft receive the
// counts behind the child segments.  The nodes that may split are listed in
// `list` (heap ids, count *n_list_d, at most n_list) or, when list is NULL,
// are nodes[0, n_list).
gbt_status partition_impl(gbt_ctx *c, const gbt_matrix *mx, const uint32_t *page, const int32_t *rows,
                          int64_t n, int32_t *position, const int32_t *slot_node, int32_t *slot_node_out,
                          DevNode *nodes, const EvalNode *list, const int32_t *n_list_d, int32_t n_list,
                          int32_t *rows_out);

}  // namespace gbt
