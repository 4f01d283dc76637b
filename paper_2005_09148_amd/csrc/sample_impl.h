// sample_impl.h -- internal interface of the sampling kernels (sample.hip)
// used by the public entry points and by the tree driver.
#pragma once

#include <algorithm>

#include "common.h"

namespace gbt {

constexpr int kCompactTile = 4096;  // rows per compaction tile
constexpr int kDigitBits = 11;
constexpr int kDigitBuckets = 1 << kDigitBits;

enum { kSrcGpair = 0, kSrcMargin = 1 };

// Which rows a sampler keeps (GBT_SAMPLE_*), given the threshold in the
// sampling state: MVS keeps a row when its key reaches T* or its draw falls
// below its key's share of T*; SGB keeps a row when its draw is below P;
// GOSS keeps the rows whose |g| key reaches the top threshold and any other
// row whose draw is below P.  all_rest: the draw always passes (p = 1).
struct SampleRule {
    int32_t mode;
    int32_t all_rest;
    uint64_t P;      // floor(p 2^64), p < 1
    double w_rest;   // GOSS: the weight of a row outside the top set
};

// Where the per-row gradient pairs come from: a float pair array, or
// recomputed from margins and labels (streamed out-of-core data).
struct SampleSrc {
    const float2 *gpair;
    const float *margin;
    const float *label;
    int32_t loss;
    int32_t pad0;
};

// Reductions over all rows land in kSpread copies, each in a 128-byte line
// of its own (block b uses copy b % kSpread), so that the blocks' atomics
// spread over kSpread cache lines instead of serializing on one; readers
// fold the copies.
constexpr int kSpread = 32;
constexpr int kLineWords = 16;  // 64-bit words per 128-byte line
typedef unsigned long long Spread[kSpread][kLineWords];

// Device-side state of one sampling + fixed-point pass.
struct SampleState {
    Spread rmax;    // max of r^2 = g^2 + lambda h^2 (double bits; >= 0)
    Spread amax;    // max key
    Spread asum;    // sum of keys (< 2^62 in total)
    Spread gmax;    // max |g'| (double bits)
    Spread hmax;    // max |h'| (double bits)
    Spread root_g;  // fixed-point sums of all training rows
    Spread root_h;
    unsigned long long C_above;    // radix descent: #keys >= upper end of the range
    unsigned long long F_below;    // radix descent: sum of keys below the range
    long long lo;                  // radix descent: range start
    long long T;                   // the threshold T*
    int32_t e_key;
    int32_t e_g, e_h;
    int32_t shift;
    int32_t nbuckets;
    int32_t levels;
    int32_t done;
    unsigned int bad;
    int32_t e_key_prev;  // e_key as the state's last use left it (kept by state_init)
    int32_t pad0;
};

// Block b's copy of a spread reduction.
__host__ __device__ inline unsigned long long *spread_at(Spread &a, unsigned b) { return &a[b % kSpread][0]; }

__host__ __device__ inline unsigned long long fold_max(const Spread &a)
{
    unsigned long long m = 0;
    for (int i = 0; i < kSpread; ++i) m = a[i][0] > m ? a[i][0] : m;
    return m;
}

__host__ __device__ inline unsigned long long fold_sum(const Spread &a)
{
    unsigned long long m = 0;
    for (int i = 0; i < kSpread; ++i) m += a[i][0];
    return m;
}

// Zeroes the state except e_key_prev, which takes the e_key the state held
// (the last tree's key exponent, the next tree's guess).
gbt_status state_init(gbt_ctx *c, SampleState *st);
// state_init's work by the threads of one block (all of them call it; no
// LDS, so that a kernel's dynamic LDS keeps its alignment).  The last word
// holds e_key_prev and the pad: thread 0 writes it from e_key first (the
// store waits for the load), then the block clears every other word.
__device__ inline void state_reset_block(SampleState *st)
{
    static_assert(sizeof(SampleState) % 8 == 0, "SampleState is zeroed in 64-bit words");
    static_assert(offsetof(SampleState, e_key_prev) == sizeof(SampleState) - 8, "e_key_prev, pad0 end the state");
    constexpr int kWords = (int)(sizeof(SampleState) / 8);
    unsigned long long *w = (unsigned long long *)st;
    if (threadIdx.x == 0) w[kWords - 1] = (unsigned long long)(uint32_t)st->e_key;
    __syncthreads();
    for (int i = threadIdx.x; i < kWords - 1; i += blockDim.x) w[i] = 0ull;
}
// keys may be NULL (recomputed on every pass).  Leaves T* in st (device).
// skip_closed: wait on the host for the closed-form test and launch the
// radix descent only when it fails (the context's pinned host buffer is
// used).
// count_mode (GOSS): K is the top count A, and T in st becomes the A-th
// largest key (INT64_MAX when A = 0) instead of the MVS threshold.
// keys_spec (with skip_closed and rmax_done): the key maximum and sum are
// already in st, formed by gradients_rmax with a guessed exponent; the
// threshold pass checks it and runs the keys pass only when it was wrong.
// defer (with skip_closed): return after the threshold's first kernel; the
// caller may queue work that reads T (it is 0, keeping every row, unless the
// closed form held) and then calls mvs_threshold_resume, after a
// synchronization of its own.
// The threshold's first step (the exponent check and the closed-form test)
// made by the selection's blocks instead of a kernel of its own.
struct ThreshFuse {
    int64_t K = 0;
    int32_t *done_host = nullptr;  // the host's flag (device address)
    int32_t check_log2n = -1;
    int32_t on = 0;
};
// fuse (deferred MVS only): the first step is left to mvs_select, with these
// arguments.
gbt_status mvs_threshold(gbt_ctx *c, const SampleSrc &src, int kind, const int64_t *keys, int64_t n,
                         double lambda, int64_t K, SampleState *st, bool skip_closed,
                         bool rmax_done = false, bool count_mode = false, bool keys_spec = false,
                         bool defer = false, ThreshFuse *fuse = nullptr);
// The rest of a deferred MVS threshold: *redo is false when the closed form
// held (T was final for the queued work), else the threshold is completed
// (the keys pass if the key exponent was guessed wrong, the radix descent)
// and the work that read T must be queued again.
gbt_status mvs_threshold_resume(gbt_ctx *c, const SampleSrc &src, int kind, const int64_t *keys, int64_t n,
                                double lambda, int64_t K, SampleState *st, bool *redo);
// Keep flags of rows [0, n) and, when tile_cnt is given, the kept count of
// each tile of kCompactTile rows.
gbt_status mvs_select(gbt_ctx *c, const SampleSrc &src, int kind, const int64_t *keys, int64_t n,
                      double lambda, SampleState *st, uint64_t seed, uint64_t iteration,
                      int64_t row_offset, uint8_t *keep, int32_t *tile_cnt, const SampleRule &rule,
                      const ThreshFuse &fuse = ThreshFuse{});
gbt_status gw_all(gbt_ctx *c, const float *gpair, int64_t n, double *gw);
// The exact fixed-point sums of all n rows' pairs (recomputed from margins
// and labels, rounded to float) into st->root_g/root_h with st->e_g/e_h,
// in two passes that keep nothing per row.
gbt_status lambda_sums(gbt_ctx *c, int32_t loss, const float *margin, const float *label, int64_t n,
                       SampleState *st);
// fx_max_done: the maxima of |g'| and |h'| are already in st (fused upstream)
gbt_status fixed_point(gbt_ctx *c, const double *gw, int64_t R, SampleState *st, int64_t *q,
                       bool fx_max_done = false);
// Gradients of all rows and, fused, the maximum of r^2 = g^2 + lambda h^2;
// with e_spec (not kNoKeySpec) also the MVS keys' maximum and sum with that
// key exponent, st->e_key = e_spec (to be checked by mvs_threshold); with
// e_spec_at (device) the exponent is read there instead.
constexpr int32_t kNoKeySpec = -0x7fffffff;
gbt_status gradients_rmax(gbt_ctx *c, int32_t loss, const float *margin, const float *label, int64_t n,
                          float *gpair, double lambda, SampleState *st, int32_t e_spec = kNoKeySpec,
                          const int32_t *e_spec_at = nullptr);
// Exclusive per-tile offsets from the per-tile counts mvs_select wrote into
// tile_off (tiles of kCompactTile rows), and the total at tile_off[tiles]
// (and at *total_host, pinned host memory, when given).
gbt_status keep_tile_offsets(gbt_ctx *c, int64_t n, int32_t *tile_off, int32_t *total_host = nullptr);
// Compaction of the kept rows among global rows [row_lo, row_hi) whose page
// words start at `words`; positions come from the tile offsets; also folds
// the maxima of |g'| and |h'| into st.  cap: the output buffers' rows; a
// tile whose kept rows would reach past it writes nothing (a compaction
// queued before the host knows the sample size, into buffers that are then
// large enough unless the sample is; the host redoes it when it was not).
// total_host (pinned, device address; rows [0, n) only): tile_off holds the
// selection's per-tile counts, not their offsets; each block sums the
// counts before its tile, and the total goes to *total_host.
gbt_status mvs_compact_tiles(gbt_ctx *c, const SampleSrc &src, int kind, int64_t n, double lambda,
                             SampleState *st, const uint8_t *keep, const int32_t *tile_off,
                             int64_t row_lo, int64_t row_hi, const uint32_t *words, int32_t row_words,
                             uint32_t *out_page, int32_t *sel, double *gw, const SampleRule &rule,
                             int64_t cap = INT64_MAX, int32_t *total_host = nullptr);
// Spins until a kernel has written a value >= 0 at *flag (pinned host
// memory); after 2 s, synchronizes the stream instead.
gbt_status wait_flag(gbt_ctx *c, volatile int32_t *flag);
// Clears the maxima of |g'| and |h'| (before a compaction is redone).
gbt_status fx_max_reset(gbt_ctx *c, SampleState *st);

}  // namespace gbt
