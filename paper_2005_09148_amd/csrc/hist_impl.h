// hist_impl.h -- internal interface of the histogram kernels (hist.hip) used
// by the tree driver, which plans the levels below the root on the device.
#pragma once

#include <vector>

#include "common.h"

namespace gbt {

struct HistWork {
    int64_t begin, end;  // rows[begin, end) of one node
    int32_t part;        // partial histogram this chunk writes
    int32_t pad0;
};

struct HistGroup {
    int32_t f0, f1;  // features [f0, f1)
    int32_t b0, b1;  // global bins [b0, b1)
    int32_t w0;      // dense: word holding the first bit of feature f0
    int32_t skip;    // dense: bit offset of feature f0 in that word
    int32_t nw;      // dense: words spanned by the group's symbols
    int32_t pad0;
};

// One built node: its partials [part0, part0 + nparts) sum into hist[slot];
// when sub_target >= 0, hist[sub_target] = parent[sub_parent] - that sum.
struct HistReduce {
    int32_t slot;
    int32_t part0;
    int32_t nparts;
    int32_t sub_parent;
    int32_t sub_target;
    int32_t pad0;
};

// Which histogram kernel a matrix uses.
enum HistKind {
    kHistSparse = 0,  // CSR pages: global-bin symbols, groups of bin ranges
    kHistDense = 1,   // dense pages, any feature up to 2560 bins
    kHistRot = 2,     // dense pages, features of at most 256 bins: lanes visit
                      // the group's features in rotated order (conflict-free LDS)
};

struct HistPlan {
    int kind;
    int threads;      // workgroup size
    int target_wgs;   // workgroups a launch aims at
    std::vector<HistGroup> groups;
    int32_t max_groups_bins;
};

// The kernel and feature groups for a matrix whose passes cover about
// rows_hint rows; choice is a GBT_HIST_* value.  GBT_E_UNSUPPORTED when a
// feature does not fit any kernel.
gbt_status hist_plan(const gbt_matrix *mx, int64_t rows_hint, int choice, HistPlan *out);

// The partition's column copy of a dense training page: m columns of
// `stride` entries, entry (f, r) the symbol of feature f in row r.  One
// byte per entry when every feature has at most 256 bins: 255 for a missing
// value, min(symbol, 254) otherwise (a reader whose split bin exceeds 254
// takes an entry of 254 from the row itself); else two bytes, the symbol.
struct ColCopy {
    void *p = nullptr;
    int64_t stride = 0;
    int32_t bytes = 0;
};

__device__ __host__ inline uint8_t col_byte(uint32_t sym, uint32_t null_sym)
{
    return (uint8_t)(sym == null_sym ? 255u : (sym < 254u ? sym : 254u));
}

// A histogram pass whose work lists live on the device.  Counts are read
// from device memory (n_work_d, n_red_d); the grids are sized by the maxima.
struct HistLaunch {
    int kind;
    const HistGroup *groups;
    int32_t n_groups;
    int32_t max_groups_bins;  // largest group, in bins
    const HistWork *work;
    const int32_t *n_work_d;
    int32_t max_work;
    const HistReduce *red;
    const int32_t *n_red_d;
    int32_t max_red;
    int64_t *partials;
    const uint8_t *slot_tbl = nullptr;  // sparse: the page's slot table by row (SlotTable::row), or NULL
    int32_t tbl_stride = 0;
    bool timed = true;  // record phase events (when the context's timing is on)
    // plain dense kernel, rows NULL (work items that cover the page's rows
    // [0, cols.stride) once): also write the page's column copy (the layout
    // split_columns makes)
    ColCopy cols;
};

// Device memory a histogram call carves its partials and plan from, in
// place of the context's workspaces (base is 256-byte aligned).
struct HistWorkspace {
    char *base;
    size_t bytes;
};

// The static scratch of the allocation-free histogram entry point: its
// device address on `device` is resolved once (hipGetSymbolAddress) with
// that device current.
gbt_status static_scratch_init(int device);

// Whether a sparse page of mx's geometry takes a slot table for G groups
// (rows of at most 255 slots and 64 words, at most 63 groups).
bool slot_table_fits(const gbt_matrix *mx, int32_t G);
// Bytes per row of the by-row layout for G groups.
inline int32_t slot_table_row_stride(int32_t G) { return (G + 1 + 3) / 4 * 4; }
// The slot table of rows [0, n) of `page` (a page of mx's geometry) for the
// groups groups_d[0, G), s_g(r) being the first slot of row r whose symbol
// is >= groups_d[g].b0 (s_G(r): the first past the last group's bins):
// row_tbl[r * slot_table_row_stride(G) + g] = s_g(r) for g <= G, and
// col_tbl[g * n + r] = s_g(r) | (s_{g+1}(r) << 8) for g < G.
gbt_status sparse_slot_table(gbt_ctx *c, const gbt_matrix *mx, const HistGroup *groups_d, int32_t G,
                             const uint32_t *page, int64_t n, uint8_t *row_tbl, uint16_t *col_tbl);

// Most bins one feature may have for the histogram kernels of a dense or a
// sparse page (one histogram group in LDS).
int32_t hist_feature_bin_limit(bool sparse);
// GBT_E_UNSUPPORTED unless every feature of mx fits that limit.
gbt_status hist_check_feature_bins(const gbt_matrix *mx);

gbt_status hist_launch_device(gbt_ctx *c, const gbt_matrix *mx, const uint32_t *page, const int64_t *q,
                              const int32_t *rows, const HistLaunch &hl, const int64_t *parent_hist,
                              int64_t *hist, unsigned long long *n_updates);

}  // namespace gbt
