// sketch_impl.h -- the batch-merged quantile sketch of Sec. 3.1 / Alg. 3 on
// the device: each batch's sorted sample keys become a per-feature summary
// that is folded into one running summary of at most S entries per feature.
//
// A summary of feature j is a list of distinct order-preserving keys
// (float_key of the values) v_1 < ... < v_k, each with a count c_i, an
// estimate of the sample values <= v_i (c_k = the values summarised).
//   batch summary: the batch's distinct values with their exact counts,
//     pruned to S entries;
//   merge(A, B): every value of A or B with c(v) = c_A(v) + c_B(v), c_X(v)
//     the count of X's last entry <= v (0 if none), pruned to S;
//   prune (k > S): for t = 1..S the entry i_t = min{ i : c_i >= ceil(tN/S) },
//     each kept once.
#pragma once

#include "common.h"

namespace gbt {

// Summaries of m features, at most S entries each: feature j's entries are
// v[j * S .. j * S + k[j]) and c[j * S ..].
struct SummarySet {
    uint32_t *v = nullptr;
    long long *c = nullptr;
    int64_t *k = nullptr;
};

// Device state of the merged sketch of one quantizer.
struct MergeSketch {
    int32_t m = 0, S = 0;
    int cur = 0;           // which of run[] holds the running summary
    SummarySet run[2];     // the running summary and the next one
    SummarySet batch;      // the current batch's summary
    uint32_t *uv = nullptr;  // the union of two summaries (2S entries per feature)
    long long *uc = nullptr;
    int32_t *pre = nullptr;  // per feature, how many of the batch's first i entries the running summary holds
    void *sort_tmp = nullptr;  // the sort's second key buffer and tile tables
    size_t sort_tmp_bytes = 0;
    std::vector<std::pair<void *, size_t>> owned;  // every allocation above
};

// Allocates the summaries (zero entries) for m features of at most S entries.
gbt_status merge_sketch_init(gbt_ctx *c, MergeSketch *ms, int32_t m, int32_t S);
void merge_sketch_free(gbt_ctx *c, MergeSketch *ms);

// One batch: keys[seg_begin[j] .. seg_begin[j] + seg_len[j]) are the batch's
// sample keys of feature j (unsorted; NaN keys 0xffffffff are missing).  The
// keys are sorted in place (segment by segment), summarised, and merged into
// the running summary.  seg_begin_h / seg_len_h are host arrays of m entries.
gbt_status merge_sketch_add(gbt_ctx *c, MergeSketch *ms, uint32_t *keys, const int64_t *seg_begin_h,
                            const int64_t *seg_len_h);

// The running summary on the host: v[j * S + i], c[j * S + i], k[j].
gbt_status merge_sketch_download(gbt_ctx *c, const MergeSketch *ms, std::vector<uint32_t> *v,
                                 std::vector<long long> *cnt, std::vector<int64_t> *k);

}  // namespace gbt
