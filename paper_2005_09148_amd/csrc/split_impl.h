// split_impl.h -- internal interface of split evaluation and partitioning
// (split.hip) used by the tree driver.
#pragma once

#include "common.h"
#include "hist_impl.h"

namespace gbt {

struct EvalParams {
    double lambda;
    double gamma;
    double mcw;
    int32_t e_g;
    int32_t e_h;
    const int32_t *e_dev;  // when set, {e_g, e_h} are read from device memory
};

// The matrix's cuts on the device, for the raw-value thresholds of splits.
struct SplitCuts {
    const float *values;
    const int32_t *ptr;
};
inline SplitCuts cuts_of(const gbt_matrix *mx) { return SplitCuts{mx->cut_values_d, mx->cut_ptr_d}; }

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
// The tree driver's fused step after a histogram pass whose features all
// have at most 256 bins: for every reduce item (count *n_red_d, at most
// max_red) and feature, sum the built node's partials into hist, write the
// sibling as parent minus it (hist may be NULL: then the sums are only
// evaluated), and evaluate the feature for both nodes (the
// EvalNode of a histogram slot is ev[slot]); cand[slot * m + feature]
// receives the candidates.  Then eval_reduce_impl picks each node's split.
gbt_status reduce_eval_impl(gbt_ctx *c, const gbt_matrix *mx, const int64_t *partials, const HistReduce *red,
                            const int32_t *n_red_d, int32_t max_red, const int64_t *parent, int64_t *hist,
                            const EvalNode *ev, const EvalParams &ep, EvalCand *cand);
// Each listed node's best split from cand (n_fblocks entries per node);
// count *n_nodes_d (at most n_nodes); decide as in eval_impl.
gbt_status eval_reduce_impl(gbt_ctx *c, const gbt_matrix *mx, const EvalCand *cand, int32_t n_fblocks,
                            const EvalNode *nodes_d, int32_t n_nodes, const int32_t *n_nodes_d, gbt_split *out_d,
                            DevNode *decide);

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

// The level's split choices made inside the partition: the candidates of the
// level's nodes (heap ids [lo, hi); a node's m candidates start at
// cand[DevNode::slot * m]).
struct LevelChoice {
    const EvalCand *cand;
    int32_t m;
    int32_t lo, hi;
};

struct PlanArgs;

// The tree driver's partition: rows[0, n) by slot_node as partition_impl,
// except that a splitting node's right rows land at the back of its segment
// in reverse slot order.  Two kernels: the first writes the left flags and,
// for each node, the tile and in-tile left count at its first and last slot
// (DevNode tile_b/left_b/tile_e/left_e); the second scatters the rows and,
// in one of its blocks, runs the level's `plan` (plan_impl.h), which turns
// those into the nodes' left counts (nleft; pleft is not written) and the
// children's records.  `order` false skips the rows' new order (rows_out and
// slot_node_out are not written) and runs the plan alone.  `root`: the root
// level, whose slots are rows 0..n-1 of node 0 (rows and slot_node are not
// read).  With `choice`, the split
// records of the level's nodes are chosen from the candidates and written
// by the first kernel (instead of by eval_reduce_impl).  With `stbl` (a
// sparse page's slot table), the search for a row's split feature looks
// only among the slots of the feature's group.  With `cols` (the page's
// column copy, split_columns), a row's split-feature symbol is read from
// its feature's column: the rows of a node ascend (or descend) along its
// segment, so a column's lines serve many of them.
gbt_status partition_rev_impl(gbt_ctx *c, const gbt_matrix *mx, const uint32_t *page, const int32_t *rows,
                              int64_t n, const int32_t *slot_node, int32_t *slot_node_out, DevNode *nodes,
                              int32_t *rows_out, const LevelChoice *choice,
                              const SlotTable *stbl, const ColCopy &cols, const PlanArgs &plan,
                              bool order, bool root);

// Whether a page of mx's geometry takes a column copy (dense, symbols of at
// most 16 bits).
bool split_columns_fit(const gbt_matrix *mx);
// The column copy (ColCopy, cols.stride >= n) of rows [0, n) of `page`
// (mx's geometry).
gbt_status split_columns(gbt_ctx *c, const gbt_matrix *mx, const uint32_t *page, int64_t n, const ColCopy &cols);
// The entry width of mx's column copy: 1 byte when every feature has at most
// 256 bins, else 2.
int32_t split_columns_bytes(const gbt_matrix *mx);

}  // namespace gbt
