// sample_impl.h -- internal interface of the sampling kernels (sample.hip)
// used by the public entry points and by the tree driver.
#pragma once

#include <algorithm>

#include "common.h"

namespace gbt {

constexpr int kDigitBits = 11;
constexpr int kDigitBuckets = 1 << kDigitBits;

enum { kSrcGpair = 0, kSrcMargin = 1 };

// Where the per-row gradient pairs come from: a float pair array, or
// recomputed from margins and labels (streamed out-of-core data).
struct SampleSrc {
    const float2 *gpair;
    const float *margin;
    const float *label;
    int32_t loss;
    int32_t pad0;
};

// Device-side state of one sampling + fixed-point pass.
struct SampleState {
    unsigned long long rmax_bits;  // max r (double bits; r >= 0)
    unsigned long long amax;       // max key
    unsigned long long asum;       // sum of keys (< 2^62)
    unsigned long long C_above;    // radix descent: #keys >= upper end of the range
    unsigned long long F_below;    // radix descent: sum of keys below the range
    long long lo;                  // radix descent: range start
    long long T;                   // the threshold T*
    unsigned long long gmax_bits, hmax_bits;
    unsigned long long root_g, root_h;  // fixed-point sums of all training rows
    int32_t e_key;
    int32_t e_g, e_h;
    int32_t shift;
    int32_t nbuckets;
    int32_t levels;
    int32_t done;
    unsigned int bad;
};

gbt_status state_init(gbt_ctx *c, SampleState *st);
// keys may be NULL (recomputed on every pass).  Leaves T* in st (device).
gbt_status mvs_threshold(gbt_ctx *c, const SampleSrc &src, int kind, const int64_t *keys, int64_t n,
                         double lambda, int64_t K, SampleState *st, SampleState *host_st);
gbt_status mvs_select(gbt_ctx *c, const SampleSrc &src, int kind, const int64_t *keys, int64_t n,
                      double lambda, const SampleState *st, uint64_t seed, uint64_t iteration,
                      int64_t row_offset, uint8_t *keep);
gbt_status mvs_compact(gbt_ctx *c, const SampleSrc &src, int kind, const int64_t *keys, int64_t n,
                       double lambda, const SampleState *st, const uint8_t *keep, const int32_t *pos,
                       const uint32_t *page, int32_t row_words, int64_t out_base, uint32_t *out_page,
                       int32_t *sel, int64_t sel_offset, double *gw);
gbt_status gw_all(gbt_ctx *c, const float *gpair, int64_t n, double *gw);
gbt_status fixed_point(gbt_ctx *c, const double *gw, int64_t R, SampleState *st, int64_t *q);

}  // namespace gbt
