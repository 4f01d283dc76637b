// hist.hip -- Alg. 1 BuildHistograms on bit-packed ELLPACK rows.
//
// Work is split two ways.  Bins: the features are cut into contiguous groups
// whose int64 (g, h) bins fit the LDS budget, with about equal bin counts.
// Rows: each built node's row segment is cut into chunks.  One workgroup owns
// one (chunk, group) pair: it accumulates the chunk's rows into its LDS
// histogram with 64-bit LDS atomics (one row per lane, the group's words
// decoded by a running bit buffer) and writes the result, with plain
// coalesced stores, as a partial histogram of that chunk.  A second kernel
// sums each node's partials into its histogram and, in the same pass, forms
// the sibling as parent minus the built child (exact integer arithmetic).
// Work items are mapped so the groups of one chunk run on the same XCD and
// share its L2 for the gradient pairs and row ids.
#include "hist_impl.h"

#include <hip/hip_ext.h>

#include <algorithm>
#include <cstring>
#include <mutex>

// Device memory of gbt_build_hist_noalloc: its partial histograms and plan.
// Every GPU the library runs on holds its own copy until the process ends;
// host code reaches it only through the address hipGetSymbolAddress gives
// on each device (the array's name is a host-side stand-in).
constexpr size_t kStaticScratchBytes = (size_t)64 << 20;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

namespace gbt {

constexpr int kHistThreads = 512;
// Sparse groups: up to 8192 bins, g then h (128 KiB of LDS), one
// 1024-thread workgroup per CU: fewer groups, so fewer reads of every row.
constexpr int kLdsBins = 10176;  // 159 KiB of int64 (g, h) sums: all of a CU's LDS
constexpr int kSparseThreads = 1024;
// value-balanced sparse groups: at least this many
constexpr int kSparseMinGroups = 16;
// Dense groups: up to 2560 bins; the h sums sit a fixed 2560 words after the
// g sums so that one address serves both atomics (an immediate offset), and
// four workgroups fit a CU's LDS.
constexpr int kDenseBins = 2560;

int32_t hist_feature_bin_limit(bool sparse) { return sparse ? kLdsBins : kDenseBins; }

gbt_status hist_check_feature_bins(const gbt_matrix *mx)
{
    const int32_t lim = hist_feature_bin_limit(mx->sparse != 0);
    for (int32_t f = 0; f < mx->m; ++f) {
        const int32_t b = mx->bin_ptr_h[f + 1] - mx->bin_ptr_h[f];
        if (b > lim)
            return set_error(GBT_E_UNSUPPORTED, "feature %d has %d bins (at most %d in a %s page)", f, b, lim,
                             mx->sparse ? "sparse" : "dense");
    }
    return GBT_OK;
}

// A dense group's bits lie within this many words from its first word (one
// 16-byte load), and it holds at most this many features.
constexpr int kGroupWords = 4;
constexpr int kMaxGroupFeat = 32;

// Zero nb entries of the g sums at sg and of the h sums at sh.
__device__ inline void lds_zero(unsigned long long *sg, unsigned long long *sh, int32_t nb)
{
    for (int t = threadIdx.x; t < nb; t += blockDim.x) {
        sg[t] = 0ull;
        sh[t] = 0ull;
    }
    __syncthreads();
}

// Write the LDS histogram as the chunk's partial and count the updates
// (cnt: this wave's count, the same in every lane).
__device__ inline void lds_flush(const unsigned long long *sg, const unsigned long long *sh,
                                 int32_t nb, longlong2 *__restrict__ dst, unsigned long long cnt,
                                 unsigned long long *__restrict__ n_updates)
{
    __shared__ unsigned long long red[16];  // one count per wave (at most 1024 threads)
    if (n_updates && (threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = cnt;
    __syncthreads();
    for (int t = threadIdx.x; t < nb; t += blockDim.x)
        dst[t] = make_longlong2((long long)sg[t], (long long)sh[t]);
    if (n_updates && threadIdx.x == 0) {
        // one atomic per block, spread over kUpdCounters addresses
        unsigned long long t = 0;
        for (int w = 0; w < (int)(blockDim.x / 64); ++w) t += red[w];
        if (t) atomicAdd(&n_updates[(blockIdx.x % kUpdCounters) * kUpdStride], t);
    }
}

// Dense rows: slot j holds feature j, W bits per symbol.  Each lane owns one
// row at a time: it fetches the next row's pair and the group's words while
// it decodes the current row.  A group's bits lie within four words from its
// first word, so the words arrive in one 16-byte load (dword aligned) and
// cost the memory pipeline one cache access per row.  After one funnel
// shift per word, feature u of the group starts at bit u*W of the window;
// with W a compile-time constant every symbol is one bit-field extract from a
// fixed register.  Null symbols are masked off; the update count comes from
// the wave's ballot.
typedef uint32_t u32x4_a4 __attribute__((ext_vector_type(4), aligned(4)));

template <int W, bool kRows>
__global__ void __launch_bounds__(kHistThreads)
    k_hist_dense(const uint32_t *__restrict__ page, int32_t row_words, uint32_t null_sym,
                 const longlong2 *__restrict__ q, const int32_t *__restrict__ rows,
                 const HistWork *__restrict__ work, const HistGroup *__restrict__ groups, int32_t n_groups,
                 const int32_t *__restrict__ n_work_d, const int32_t *__restrict__ bin_ptr, int64_t total_bins,
                 longlong2 *__restrict__ partials, unsigned long long *__restrict__ n_updates, ColCopy cols)
{
    extern __shared__ unsigned long long lds[];
    const uint32_t active = n_work_d ? (uint32_t)(*n_work_d * n_groups) : gridDim.x;
    if (blockIdx.x >= active) return;
    const uint32_t L = xcd_remap(blockIdx.x, active);
    const HistWork wk = work[L / n_groups];
    const HistGroup gr = groups[L % n_groups];
    const int32_t nb = gr.b1 - gr.b0, nf = gr.f1 - gr.f0;
    unsigned long long *sg = lds, *sh = lds + kDenseBins;
    constexpr uint32_t kMask = (1u << W) - 1u;
    constexpr int kMaxF = (kGroupWords * 32 / W) < kMaxGroupFeat ? (kGroupWords * 32 / W) : kMaxGroupFeat;
    // the 16-byte window starts at the group's first word, or ends at the
    // row's last word when the group sits in the row's last three words
    const int32_t ws = gr.w0 < row_words - kGroupWords ? gr.w0 : row_words - kGroupWords;
    const int32_t dw = gr.w0 - ws;  // 0..3 words, the same in every lane
    // byte address of each feature's first g sum (uniform)
    char *base[kMaxF];
#pragma unroll
    for (int u = 0; u < kMaxF; ++u) base[u] = (char *)(sg + (u < nf ? bin_ptr[gr.f0 + u] - gr.b0 : 0));
    lds_zero(sg, sh, nb);

    unsigned int cnt = 0;  // this wave's updates
    int64_t i = wk.begin + threadIdx.x;
    longlong2 qn = make_longlong2(0, 0);
    u32x4_a4 wn = {0u, 0u, 0u, 0u};
    auto fetch = [&](int64_t ii) {
        const int64_t r = kRows ? (int64_t)rows[ii] : ii;
        qn = q[r];
        wn = *(const u32x4_a4 *)(page + r * row_words + ws);
    };
    if (i < wk.end) fetch(i);
    for (; i < wk.end; i += kHistThreads) {
        const unsigned long long qg = (unsigned long long)qn.x, qh = (unsigned long long)qn.y;
        uint32_t y[kGroupWords + 1] = {wn.x, wn.y, wn.z, wn.w, 0u};
        if (dw) {  // uniform: drop the dw words before the group
#pragma unroll
            for (int k = 0; k < kGroupWords; ++k) {
                const uint32_t y1 = k + 1 < kGroupWords ? y[k + 1] : 0u, y2 = k + 2 < kGroupWords ? y[k + 2] : 0u,
                               y3 = k + 3 < kGroupWords ? y[k + 3] : 0u;
                y[k] = dw == 1 ? y1 : (dw == 2 ? y2 : y3);
            }
        }
        // a[k] = bits [32k + skip, 32k + skip + 32) of the group's words
        uint32_t a[kGroupWords + 1];
#pragma unroll
        for (int k = 0; k < kGroupWords; ++k) a[k] = __builtin_amdgcn_alignbit(y[k + 1], y[k], (uint32_t)gr.skip);
        a[kGroupWords] = 0u;
        if (i + kHistThreads < wk.end) fetch(i + kHistThreads);
#pragma unroll
        for (int u = 0; u < kMaxF; ++u) {
            if (u < nf) {
                const int bit = u * W, k = bit >> 5, sft = bit & 31;
                uint32_t sym;
                if (sft + W <= 32)
                    sym = (a[k] >> sft) & kMask;
                else
                    sym = __builtin_amdgcn_alignbit(a[k + 1], a[k], (uint32_t)sft) & kMask;
                const bool ok = sym != null_sym;
                cnt += (unsigned int)__popcll(__ballot(ok));
                // a pass over the page in row order also writes the column
                // copy: entry (f, row) for each feature f of the group
                if (!kRows && cols.p) {
                    const int64_t e = (int64_t)(gr.f0 + u) * cols.stride + i;
                    if (cols.bytes == 1)
                        ((uint8_t *)cols.p)[e] = col_byte(sym, null_sym);
                    else
                        ((uint16_t *)cols.p)[e] = (uint16_t)sym;
                }
                if (ok) {
                    unsigned long long *pg = (unsigned long long *)(base[u] + sym * 8u);
                    atomicAdd(pg, qg);
                    atomicAdd(pg + kDenseBins, qh);
                }
            }
        }
    }
    lds_flush(sg, sh, nb, partials + (int64_t)wk.part * total_bins + gr.b0, cnt, n_updates);
}

// ---------------------------------------------------------------- rotated
// Dense rows whose features have at most 256 bins (symbols of at most 9
// bits).  One row per lane; a group holds at most 16 features whose bits lie
// within four words from its first word (one 16-byte load, as in the plain
// kernel).  The LDS sums are 256 bin rows of 16 columns, column c holding
// one feature, so the address of (feature, bin) is bin*128 + column*8 and
// its LDS bank pair is set by the column and the bin's parity.  Lane l
// visits the group's features starting at feature l mod nf: in every atomic
// the 64 lanes spread over the columns instead of colliding at random bins
// of one feature.  The rotation is applied once per row: the group's bit
// string S (nf*W bits) is doubled to D = S | S << nf*W (a shift that is the
// same in every lane), and each lane takes D >> (c0*W), so each step's
// symbol is still a fixed bit field.  Two workgroups share a CU.
constexpr int kRotThreads = 512;
constexpr int kRotCols = 16;
constexpr int kRotBins = 256;
constexpr int kRotMaxW = 9;
// rows per tree level from which the rotated kernel is chosen by default
constexpr int64_t kRotMinRows = (int64_t)2 << 20;

__device__ inline uint32_t pick(bool c, uint32_t a, uint32_t b) { return c ? a : b; }

// D[k] = S[k] | word k of (S << nfw), for the word part lq of the shift
template <int lq>
__device__ inline void shl_words(const uint32_t S[kGroupWords], uint32_t sh, uint32_t D[2 * kGroupWords])
{
#pragma unroll
    for (int k = 0; k < 2 * kGroupWords; ++k) {
        const int j = k - lq;
        const uint32_t hi = (j + 1 >= 0 && j + 1 < kGroupWords) ? S[j + 1] : 0u;
        const uint32_t lo = (j >= 0 && j < kGroupWords) ? S[j] : 0u;
        D[k] = (k < kGroupWords ? S[k] : 0u) | __builtin_amdgcn_alignbit(hi, lo, sh);
    }
}

template <int W, bool kRows>
__global__ void __launch_bounds__(kRotThreads)
    k_hist_rot(const uint32_t *__restrict__ page, int32_t row_words, uint32_t null_sym,
               const longlong2 *__restrict__ q, const int32_t *__restrict__ rows,
               const HistWork *__restrict__ work, const HistGroup *__restrict__ groups, int32_t n_groups,
               const int32_t *__restrict__ n_work_d, const int32_t *__restrict__ bin_ptr, int64_t total_bins,
               longlong2 *__restrict__ partials, unsigned long long *__restrict__ n_updates)
{
    extern __shared__ unsigned long long lds[];
    constexpr int kH = kRotBins * kRotCols;  // h sums follow the g sums
    const uint32_t active = n_work_d ? (uint32_t)(*n_work_d * n_groups) : gridDim.x;
    if (blockIdx.x >= active) return;
    const uint32_t L = xcd_remap(blockIdx.x, active);
    const HistWork wk = work[L / n_groups];
    const HistGroup gr = groups[L % n_groups];
    const int32_t nf = gr.f1 - gr.f0;
    constexpr uint32_t kMask = (1u << W) - 1u;
    constexpr int kMaxF = (kGroupWords * 32 / W) < kRotCols ? (kGroupWords * 32 / W) : kRotCols;

    for (int t = threadIdx.x; t < 2 * kH; t += kRotThreads) lds[t] = 0ull;
    __syncthreads();

    const int lane = threadIdx.x & 63;
    const int c0 = lane % nf;
    // LDS byte address of the column visited at step u
    uint32_t colb[kMaxF];
#pragma unroll
    for (int u = 0; u < kMaxF; ++u) {
        int c = c0 + u;
        c = c >= nf ? c - nf : c;
        c = c >= nf ? c - nf : c;
        colb[u] = (uint32_t)c * 8u;
    }
    const int32_t ws = gr.w0 < row_words - kGroupWords ? gr.w0 : row_words - kGroupWords;
    const int32_t dw = gr.w0 - ws;  // words before the group in the window (uniform)
    const int nfw = nf * W;         // bits of the group, at most 128
    // bits of S: keep[k] masks word k
    uint32_t keep[kGroupWords];
#pragma unroll
    for (int k = 0; k < kGroupWords; ++k) {
        const int lo = k * 32;
        keep[k] = nfw >= lo + 32 ? 0xffffffffu : (nfw <= lo ? 0u : ((1u << (nfw - lo)) - 1u));
    }
    // D = S | S << nfw: word k of S << nfw is bits [32k - nfw, 32k - nfw + 32)
    // of S, a funnel of S[k - lq + 1] and S[k - lq] by (-nfw) mod 32
    const int lq = (nfw + 31) >> 5;
    const uint32_t sh_nfw = (uint32_t)(-nfw) & 31u;
    // lane's rotation: D >> rho
    const int rho = c0 * W, rw = rho >> 5, rb = rho & 31;
    char *const base = (char *)lds;

    unsigned int cnt = 0;  // this wave's updates
    int64_t i = wk.begin + threadIdx.x;
    longlong2 qn = make_longlong2(0, 0);
    u32x4_a4 wn = {0u, 0u, 0u, 0u};
    auto fetch = [&](int64_t ii) {
        const int64_t r = kRows ? (int64_t)rows[ii] : ii;
        qn = q[r];
        wn = *(const u32x4_a4 *)(page + r * row_words + ws);
    };
    if (i < wk.end) fetch(i);
    for (; i < wk.end; i += kRotThreads) {
        const unsigned long long qg = (unsigned long long)qn.x, qh = (unsigned long long)qn.y;
        uint32_t y[kGroupWords + 1] = {wn.x, wn.y, wn.z, wn.w, 0u};
        if (i + kRotThreads < wk.end) fetch(i + kRotThreads);
        if (dw) {  // uniform: drop the dw words before the group
#pragma unroll
            for (int k = 0; k < kGroupWords; ++k) {
                const uint32_t y1 = k + 1 < kGroupWords ? y[k + 1] : 0u, y2 = k + 2 < kGroupWords ? y[k + 2] : 0u,
                               y3 = k + 3 < kGroupWords ? y[k + 3] : 0u;
                y[k] = dw == 1 ? y1 : (dw == 2 ? y2 : y3);
            }
        }
        // S: the group's bit string from bit 0, zero above nfw
        uint32_t S[kGroupWords];
#pragma unroll
        for (int k = 0; k < kGroupWords; ++k)
            S[k] = __builtin_amdgcn_alignbit(y[k + 1], y[k], (uint32_t)gr.skip) & keep[k];
        // D, eight words; the shift by nfw is the same in every lane (a scalar branch)
        uint32_t D[2 * kGroupWords];
        switch (lq) {
            case 0: shl_words<0>(S, sh_nfw, D); break;
            case 1: shl_words<1>(S, sh_nfw, D); break;
            case 2: shl_words<2>(S, sh_nfw, D); break;
            case 3: shl_words<3>(S, sh_nfw, D); break;
            default: shl_words<4>(S, sh_nfw, D); break;
        }
        // R = D >> rho (word shift rw = 0..3 by two selects, then the bit shift)
        uint32_t s1[7], s2[5], R[kGroupWords + 1];
#pragma unroll
        for (int k = 0; k < 7; ++k) s1[k] = pick(rw & 1, D[k + 1], D[k]);
#pragma unroll
        for (int k = 0; k < 5; ++k) s2[k] = pick(rw & 2, s1[k + 2], s1[k]);
#pragma unroll
        for (int k = 0; k < kGroupWords; ++k) R[k] = __builtin_amdgcn_alignbit(s2[k + 1], s2[k], (uint32_t)rb);
        R[kGroupWords] = 0u;
#pragma unroll
        for (int u = 0; u < kMaxF; ++u) {
            if (u < nf) {
                const int bit = u * W, k = bit >> 5, sft = bit & 31;
                uint32_t sym;
                if (sft + W <= 32)
                    sym = (R[k] >> sft) & kMask;
                else
                    sym = __builtin_amdgcn_alignbit(R[k + 1], R[k], (uint32_t)sft) & kMask;
                // symbols outside the bin range (only in a malformed page) are skipped
                const bool ok = sym != null_sym && sym < (uint32_t)kRotBins;
                cnt += (unsigned int)__popcll(__ballot(ok));
                if (ok) {
                    unsigned long long *pg = (unsigned long long *)(base + colb[u] + sym * (kRotCols * 8u));
                    atomicAdd(pg, qg);
                    atomicAdd(pg + kH, qh);
                }
            }
        }
    }
    // the update count: one atomic per wave (the LDS is all histogram)
    if (n_updates && lane == 0 && cnt)
        atomicAdd(&n_updates[((blockIdx.x * (kRotThreads / 64) + (threadIdx.x >> 6)) % kUpdCounters) * kUpdStride],
                  (unsigned long long)cnt);
    // partial of this chunk: feature f's bins are column f of the bin rows;
    // consecutive lanes read consecutive columns (no bank conflicts), and the
    // four bins of a wave's 64 lanes write 64-byte runs per feature
    __syncthreads();
    longlong2 *dst = partials + (int64_t)wk.part * total_bins;
    for (int t = threadIdx.x; t < kRotBins * kRotCols; t += kRotThreads) {
        const int b = t / kRotCols, ff = t - b * kRotCols;
        if (ff < nf) {
            const int32_t g0 = bin_ptr[gr.f0 + ff];
            if (g0 + b < bin_ptr[gr.f0 + ff + 1]) {
                const unsigned long long *src = lds + t;
                dst[g0 + b] = make_longlong2((long long)src[0], (long long)src[kH]);
            }
        }
    }
}

// Sparse rows: the row's present features in ascending order as global
// bins, null padded; the group keeps the symbols in its bin range.  A lane
// finds the row's first symbol of the group by binary search (the symbols
// are ascending) and reads on until the group's end.
__device__ inline uint32_t sparse_symbol(const uint32_t *__restrict__ row, int32_t s, int32_t w, uint32_t mask)
{
    const uint32_t bit = (uint32_t)s * (uint32_t)w, k = bit >> 5, sh = bit & 31u;
    uint32_t v = row[k] >> sh;
    if (sh + (uint32_t)w > 32u) v |= row[k + 1] << (32u - sh);
    return v & mask;
}

template <bool kRows>
__global__ void __launch_bounds__(kSparseThreads)
    k_hist_sparse(const uint32_t *__restrict__ page, int32_t row_words, int32_t w, uint32_t mask,
                  int32_t stride, const longlong2 *__restrict__ q, const int32_t *__restrict__ rows,
                  const HistWork *__restrict__ work, const HistGroup *__restrict__ groups,
                  int32_t n_groups, const int32_t *__restrict__ n_work_d, int64_t total_bins,
                  longlong2 *__restrict__ partials, unsigned long long *__restrict__ n_updates,
                  const uint8_t *__restrict__ slot_tbl, int32_t tbl_stride)
{
    extern __shared__ unsigned long long lds[];
    const uint32_t active = n_work_d ? (uint32_t)(*n_work_d * n_groups) : gridDim.x;
    if (blockIdx.x >= active) return;
    const uint32_t L = xcd_remap(blockIdx.x, active);
    const HistWork wk = work[L / n_groups];
    const int32_t gi = (int32_t)(L % n_groups);
    const HistGroup gr = groups[gi];
    const int32_t nb = gr.b1 - gr.b0;
    unsigned long long *sg = lds, *sh = lds + nb;
    lds_zero(sg, sh, nb);
    unsigned long long cnt = 0;
    const uint32_t b0 = (uint32_t)gr.b0, b1 = (uint32_t)gr.b1;
    for (int64_t i = wk.begin + threadIdx.x; i < wk.end; i += kSparseThreads) {
        const int64_t r = kRows ? (int64_t)rows[i] : i;
        const uint32_t *p = page + r * row_words;
        int32_t a = 0, e = stride;  // the slots to read: [a, e)
        if (slot_tbl) {
            const uint8_t *t = slot_tbl + r * tbl_stride + gi;
            a = t[0];
            e = t[1];
            if (a >= e) continue;  // no symbol of the group in this row
        } else {
            int32_t x = 0, y = stride;  // first slot whose symbol is >= b0
            while (x < y) {
                const int32_t mid = (x + y) >> 1;
                if (sparse_symbol(p, mid, w, mask) < b0)
                    x = mid + 1;
                else
                    y = mid;
            }
            a = x;
        }
        const longlong2 qq = q[r];
        const unsigned long long qg = (unsigned long long)qq.x, qh = (unsigned long long)qq.y;
        for (int32_t s = a; s < e; ++s) {
            const uint32_t sym = sparse_symbol(p, s, w, mask);
            if (sym >= b1) break;  // ascending; padding is the largest symbol
            if (sym < b0) continue;  // only in a page whose symbols are not ascending
            const int32_t idx = (int32_t)(sym - b0);
            atomicAdd(&sg[idx], qg);
            atomicAdd(&sh[idx], qh);
            ++cnt;
        }
    }
    // the flush takes one count per wave
    for (int d = 32; d > 0; d >>= 1) cnt += __shfl_xor(cnt, d, 64);
    lds_flush(sg, sh, nb, partials + (int64_t)wk.part * total_bins + gr.b0, cnt, n_updates);
}

// Slot table of a sparse page: a thread per row loads the row's words into
// registers with 16-byte loads (all in flight at once) and reads its
// symbols in order through a 64-bit bit buffer (the symbol width is the
// same for every row, so the decode loop is uniform); a symbol at or past
// the current group's end opens the next groups.  Each thread keeps its
// row's group starts in LDS and writes the row's entry of every group's
// 2-byte column (consecutive threads, consecutive rows).
constexpr int kTblThreads = 256;
constexpr int kTblMaxStride = 64;  // group starts per row (groups + 1)
constexpr int kTblMaxWords = 64;   // row words held in registers

typedef uint32_t u32x4_t4 __attribute__((ext_vector_type(4), aligned(4)));

template <int kMaxWords>
__global__ void __launch_bounds__(kTblThreads)
    k_sparse_slot_table(const uint32_t *__restrict__ page, int64_t n, int32_t row_words, int32_t stride, int32_t w,
                        uint32_t mask, const HistGroup *__restrict__ groups, int32_t G, uint8_t *__restrict__ row_tbl,
                        int32_t rs, uint16_t *__restrict__ col_tbl)
{
    __shared__ uint32_t ends[kTblMaxStride];
    constexpr int kPitch = kTblMaxStride + 4;  // 17 words: the threads' bytes on distinct banks
    __shared__ uint8_t out_l[kTblThreads * kPitch];
    uint8_t *o = out_l + threadIdx.x * kPitch;
    for (int32_t g = threadIdx.x; g < kTblMaxStride; g += kTblThreads)
        ends[g] = g < G ? (uint32_t)groups[g].b1 : 0xffffffffu;
    const int64_t r0 = (int64_t)blockIdx.x * kTblThreads;
    const int32_t nr = (int32_t)min<int64_t>(kTblThreads, n - r0);
    uint32_t wd[kMaxWords];
    if ((int32_t)threadIdx.x < nr) {
        const uint32_t *row = page + (r0 + threadIdx.x) * row_words;
#pragma unroll
        for (int q = 0; q < kMaxWords / 4; ++q) {
            if (4 * q + 4 <= row_words) {
                const u32x4_t4 v = *(const u32x4_t4 *)(row + 4 * q);
                wd[4 * q] = v.x;
                wd[4 * q + 1] = v.y;
                wd[4 * q + 2] = v.z;
                wd[4 * q + 3] = v.w;
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j) wd[4 * q + j] = 4 * q + j < row_words ? row[4 * q + j] : 0u;
            }
        }
    }
    __syncthreads();
    if ((int32_t)threadIdx.x < nr) {
        uint64_t buf = 0;
        int32_t nb = 0, s = 0, g = 0;
        uint32_t end = ends[0];
        o[0] = 0;
#pragma unroll
        for (int k = 0; k < kMaxWords; ++k) {
            if (k < row_words) {
                buf |= (uint64_t)wd[k] << nb;
                nb += 32;
                while (nb >= w && s < stride) {
                    const uint32_t v = (uint32_t)buf & mask;
                    buf >>= w;
                    nb -= w;
                    while (v >= end && g < G) {
                        o[++g] = (uint8_t)s;
                        end = ends[g];
                    }
                    ++s;
                }
            }
        }
        while (g < G) o[++g] = (uint8_t)stride;
        // the row's entry (word stores), then its place in each group's
        // 2-byte column (consecutive threads, consecutive rows)
        uint32_t *dr = (uint32_t *)(row_tbl + (r0 + threadIdx.x) * rs);
        for (int32_t k = 0; k < rs / 4; ++k) dr[k] = ((const uint32_t *)o)[k];
        uint16_t *dc = col_tbl + r0 + threadIdx.x;
        for (int32_t k = 0; k < G; ++k) dc[(int64_t)k * n] = (uint16_t)(o[k] | (o[k + 1] << 8));
    }
}

bool slot_table_fits(const gbt_matrix *mx, int32_t G)
{
    return mx->sparse && G >= 1 && G < kTblMaxStride && mx->stride <= 255 && mx->row_words <= kTblMaxWords;
}

gbt_status sparse_slot_table(gbt_ctx *c, const gbt_matrix *mx, const HistGroup *groups_d, int32_t G,
                             const uint32_t *page, int64_t n, uint8_t *row_tbl, uint16_t *col_tbl)
{
    if (!slot_table_fits(mx, G)) return set_error(GBT_E_INVALID, "the page takes no slot table (%d groups)", G);
    if (n <= 0) return GBT_OK;
    const uint32_t mask = mx->w >= 32 ? 0xffffffffu : ((1u << mx->w) - 1u);
    const unsigned grid = (unsigned)((n + kTblThreads - 1) / kTblThreads);
    const int32_t rw = mx->row_words;
#define GBT_TBL(MW)                                                                                      \
    k_sparse_slot_table<MW><<<grid, kTblThreads, 0, c->stream>>>(page, n, rw, mx->stride, mx->w, mask, \
                                                                 groups_d, G, row_tbl,                 \
                                                                 slot_table_row_stride(G), col_tbl)
    if (rw <= 8)
        GBT_TBL(8);
    else if (rw <= 16)
        GBT_TBL(16);
    else if (rw <= 32)
        GBT_TBL(32);
    else
        GBT_TBL(64);
#undef GBT_TBL
    GBT_LAUNCHED();
    return GBT_OK;
}

// Sums each built node's partials into its histogram and, in the same pass,
// writes the sibling as parent minus that sum.  A block covers 64 bins; its
// four waves sum every fourth partial and fold through LDS, so even a single
// node's reduction spreads over total_bins / 64 blocks.
constexpr int kRedBins = 64;
constexpr int kRedSplit = 4;

__global__ void __launch_bounds__(kRedBins * kRedSplit)
    k_hist_reduce(const longlong2 *__restrict__ partials, const HistReduce *__restrict__ red,
                  const int32_t *__restrict__ n_red_d, const longlong2 *__restrict__ parent,
                  longlong2 *__restrict__ hist, int64_t total_bins)
{
    if (n_red_d && (int32_t)blockIdx.y >= *n_red_d) return;
    __shared__ long long sg[kRedSplit][kRedBins], sh[kRedSplit][kRedBins];
    const HistReduce rd = red[blockIdx.y];
    const int lane = threadIdx.x % kRedBins, s = threadIdx.x / kRedBins;
    const int64_t b = (int64_t)blockIdx.x * kRedBins + lane;
    long long g = 0, h = 0;
    if (b < total_bins) {
        for (int32_t k = s; k < rd.nparts; k += kRedSplit) {
            const longlong2 v = partials[(int64_t)(rd.part0 + k) * total_bins + b];
            g += v.x;
            h += v.y;
        }
    }
    sg[s][lane] = g;
    sh[s][lane] = h;
    __syncthreads();
    if (s == 0 && b < total_bins) {
        for (int t = 1; t < kRedSplit; ++t) {
            g += sg[t][lane];
            h += sh[t][lane];
        }
        hist[(int64_t)rd.slot * total_bins + b] = make_longlong2(g, h);
        if (rd.sub_target >= 0) {
            const longlong2 pv = parent[(int64_t)rd.sub_parent * total_bins + b];
            hist[(int64_t)rd.sub_target * total_bins + b] = make_longlong2(pv.x - g, pv.y - h);
        }
    }
}

// Feature groups: contiguous features with about equal bin counts, each
// group within its kernel's limits (LDS bins; for dense rows also the words
// and features one lane decodes).
static bool dense_groups(const gbt_matrix *mx, int64_t max_bins, int max_feat, int max_words,
                         std::vector<HistGroup> *out)
{
    out->clear();
    const int64_t tb = mx->total_bins;
    const int64_t G = std::max<int64_t>(
        {(int64_t)1, (tb + max_bins - 1) / max_bins, ((int64_t)mx->m + max_feat - 1) / max_feat});
    auto fits = [&](int32_t f0, int32_t f1) {
        const int64_t b0 = (int64_t)f0 * mx->w, b1 = (int64_t)f1 * mx->w;
        const int32_t nw = (int32_t)((b1 + 31) / 32 - b0 / 32);
        return nw <= max_words && f1 - f0 <= max_feat && mx->bin_ptr_h[f1] - mx->bin_ptr_h[f0] <= max_bins;
    };
    int32_t f0 = 0;
    int64_t left = G;  // groups still to form; each takes an equal share of what remains
    while (f0 < mx->m) {
        if (!fits(f0, f0 + 1)) return false;
        const int64_t share = std::max<int64_t>(1, left--);
        const int64_t target_bins = (tb - mx->bin_ptr_h[f0] + share - 1) / share;
        const int64_t target_feat = (mx->m - f0 + share - 1) / share;
        int32_t f1 = f0 + 1;
        while (f1 < mx->m && fits(f0, f1 + 1) && mx->bin_ptr_h[f1 + 1] - mx->bin_ptr_h[f0] <= target_bins &&
               f1 + 1 - f0 <= target_feat)
            ++f1;
        HistGroup g;
        g.f0 = f0;
        g.f1 = f1;
        g.b0 = mx->bin_ptr_h[f0];
        g.b1 = mx->bin_ptr_h[f1];
        const int64_t bit = (int64_t)f0 * mx->w;
        g.w0 = (int32_t)(bit >> 5);
        g.skip = (int32_t)(bit & 31);
        g.nw = (int32_t)(((int64_t)f1 * mx->w + 31) / 32 - bit / 32);
        g.pad0 = 0;
        out->push_back(g);
        f0 = f1;
    }
    return true;
}

// Sparse groups: contiguous features of at most kLdsBins bins.  With the
// features' value counts known, a group also holds at most twice an equal
// share (over max(groups by bins, kSparseMinGroups)) of the values, so that
// popular features make small groups and no group's workgroups carry most
// of the updates; otherwise the groups take equal shares of the bins.
static void sparse_groups(const gbt_matrix *mx, std::vector<HistGroup> *out)
{
    out->clear();
    const int64_t tb = mx->total_bins;
    const int64_t G = std::max<int64_t>(1, (tb + kLdsBins - 1) / kLdsBins);
    const bool counts = (int32_t)mx->feat_count_h.size() == mx->m;
    int64_t total = 0;
    if (counts)
        for (int64_t v : mx->feat_count_h) total += v;
    const int64_t Gc = std::max<int64_t>(G, kSparseMinGroups);
    const int64_t target = counts ? kLdsBins : (tb + G - 1) / G;
    const int64_t target_cnt = counts ? std::max<int64_t>(1, 2 * ((total + Gc - 1) / Gc)) : INT64_MAX;
    int32_t f0 = 0;
    while (f0 < mx->m) {
        int32_t f1 = f0 + 1;
        int64_t cnt = counts ? mx->feat_count_h[f0] : 0;
        while (f1 < mx->m && mx->bin_ptr_h[f1 + 1] - mx->bin_ptr_h[f0] <= target &&
               (!counts || cnt + mx->feat_count_h[f1] <= target_cnt)) {
            if (counts) cnt += mx->feat_count_h[f1];
            ++f1;
        }
        HistGroup g{f0, f1, mx->bin_ptr_h[f0], mx->bin_ptr_h[f1], 0, 0, 0, 0};
        out->push_back(g);
        f0 = f1;
    }
}

gbt_status hist_plan(const gbt_matrix *mx, int64_t rows_hint, int choice, HistPlan *out)
{
    out->groups.clear();
    int32_t max_feature_bins = 0;
    for (int32_t f = 0; f < mx->m; ++f)
        max_feature_bins = std::max(max_feature_bins, mx->bin_ptr_h[f + 1] - mx->bin_ptr_h[f]);
    if (mx->sparse) {
        if (max_feature_bins > kLdsBins)
            return set_error(GBT_E_UNSUPPORTED, "a feature has %d bins (at most %d)", max_feature_bins,
                             kLdsBins);
        out->kind = kHistSparse;
        out->threads = kSparseThreads;
        out->target_wgs = 2 * kCUs;  // two rounds of one workgroup per CU
        sparse_groups(mx, &out->groups);
    } else {
        if (mx->w < 1 || mx->w > 12 || max_feature_bins > kDenseBins)
            return set_error(GBT_E_UNSUPPORTED, "a feature has %d bins (at most %d in a dense page)",
                             max_feature_bins, kDenseBins);
        // the rotated kernel pays off on large passes; smaller ones keep more
        // workgroups per CU with the plain kernel
        const bool want_rot = choice == GBT_HIST_ROTATED || (choice == GBT_HIST_AUTO && rows_hint >= kRotMinRows);
        if (want_rot && max_feature_bins <= kRotBins && mx->w <= kRotMaxW &&
            dense_groups(mx, (int64_t)kRotBins * kRotCols, kRotCols, kGroupWords, &out->groups)) {
            out->kind = kHistRot;
            out->threads = kRotThreads;
            out->target_wgs = 2 * kCUs;  // two workgroups per CU
        } else {
            if (!dense_groups(mx, kDenseBins, kMaxGroupFeat, kGroupWords, &out->groups))
                return set_error(GBT_E_UNSUPPORTED, "no feature grouping fits the histogram kernel");
            out->kind = kHistDense;
            out->threads = kHistThreads;
            out->target_wgs = 2 * kCUs;
        }
    }
    out->max_groups_bins = 0;
    for (auto &g : out->groups) out->max_groups_bins = std::max(out->max_groups_bins, g.b1 - g.b0);
    return GBT_OK;
}

gbt_status build_hist_impl(gbt_ctx *c, const gbt_matrix *mx, const uint32_t *page, const int64_t *q,
                           const int32_t *rows, const gbt_seg *build, int32_t n_build,
                           const gbt_sub *sub, int32_t n_sub, const int64_t *parent_hist,
                           int64_t *hist, gbt_tree_stats *stats, const HistWorkspace *ws)
{
    const int64_t tb = mx->total_bins;
    if (tb == 0 || n_build == 0) {
        GBT_CHECK(n_sub == 0, "a subtraction needs its built sibling in the same call");
        return GBT_OK;
    }
    int64_t total_rows = 0;
    for (int32_t k = 0; k < n_build; ++k) total_rows += std::max<int64_t>(0, build[k].end - build[k].begin);
    HistPlan hp;
    GBT_TRY(hist_plan(mx, total_rows, c->hist_kernel, &hp));
    const std::vector<HistGroup> &groups = hp.groups;
    const int32_t G = (int32_t)groups.size();
    // chunks: at most the kernel's workgroup target over all groups (each node
    // adds at most one chunk), at least 2048 rows each
    const int64_t items = std::max<int64_t>(1, hp.target_wgs / G - n_build);
    int64_t chunk = (total_rows + items - 1) / items;
    chunk = std::max<int64_t>(chunk, 2048);
    auto al = [](size_t b) { return (b + 255) / 256 * 256; };
    if (ws) {
        // the partials and the plan must fit the given workspace: fewer,
        // longer chunks when the usual ones would not (each non-empty node
        // needs at least one)
        int64_t nonempty = 0, longest = 0;
        for (int32_t k = 0; k < n_build; ++k) {
            const int64_t len = std::max<int64_t>(0, build[k].end - build[k].begin);
            nonempty += len > 0;
            longest = std::max(longest, len);
        }
        const size_t fixed = al((size_t)G * sizeof(HistGroup)) + al((size_t)n_build * sizeof(HistReduce)) + 4 * 256;
        const size_t per_part = (size_t)tb * 16 + sizeof(HistWork);
        const int64_t pmax = ws->bytes > fixed ? (int64_t)((ws->bytes - fixed) / per_part) : 0;
        if (pmax < nonempty)
            return set_error(GBT_E_INVALID,
                             "%lld non-empty nodes of %lld bins need %zu bytes of scratch; the static scratch "
                             "holds %zu",
                             (long long)nonempty, (long long)tb, fixed + (size_t)nonempty * per_part, ws->bytes);
        if (nonempty > 0) {
            const int64_t room = pmax - nonempty;
            chunk = std::max(chunk, room > 0 ? (total_rows + room - 1) / room : longest);
        }
    }
    std::vector<HistWork> work;
    std::vector<HistReduce> red;
    int32_t nparts = 0;
    for (int32_t k = 0; k < n_build; ++k) {
        HistReduce rd{build[k].node_slot, nparts, 0, -1, -1, 0};
        for (int64_t b = build[k].begin; b < build[k].end; b += chunk) {
            work.push_back({b, std::min(build[k].end, b + chunk), nparts, 0});
            ++nparts;
            ++rd.nparts;
        }
        red.push_back(rd);
    }
    for (int32_t s = 0; s < n_sub; ++s) {
        int32_t k = 0;
        while (k < n_build && build[k].node_slot != sub[s].built_slot) ++k;
        GBT_CHECK(k < n_build, "subtraction %d names slot %d, which is not built", s, sub[s].built_slot);
        GBT_CHECK(red[k].sub_target < 0, "slot %d is the built child of two subtractions", sub[s].built_slot);
        red[k].sub_parent = sub[s].parent_slot;
        red[k].sub_target = sub[s].target_slot;
    }

    // upload the plan: groups | work | reduce items
    size_t o_w = al((size_t)G * sizeof(HistGroup));
    size_t o_r = o_w + al(std::max<size_t>(work.size(), 1) * sizeof(HistWork));
    size_t bytes = o_r + red.size() * sizeof(HistReduce) + 256;
    const size_t part_bytes = (size_t)std::max(nparts, 1) * tb * 16;
    char *plan;
    longlong2 *partials = nullptr;
    if (ws) {
        // partials first, then the plan, in the caller's workspace
        if (al(part_bytes) + bytes > ws->bytes)
            return set_error(GBT_E_INVALID, "the histogram plan needs %zu bytes of scratch; the static scratch holds %zu",
                             al(part_bytes) + bytes, ws->bytes);
        partials = (longlong2 *)ws->base;
        plan = ws->base + al(part_bytes);
    } else {
        GBT_TRY(scratch_t(c, kScrWork, bytes, &plan));
        GBT_TRY(scratch(c, kScrPartials, part_bytes, (void **)&partials));
    }
    std::vector<char> h(bytes);
    memcpy(h.data(), groups.data(), G * sizeof(HistGroup));
    if (!work.empty()) memcpy(h.data() + o_w, work.data(), work.size() * sizeof(HistWork));
    memcpy(h.data() + o_r, red.data(), red.size() * sizeof(HistReduce));
    GBT_HIP(hipMemcpyAsync(plan, h.data(), bytes, hipMemcpyHostToDevice, c->stream));
    const HistGroup *groups_d = (const HistGroup *)plan;
    const HistWork *work_d = (const HistWork *)(plan + o_w);
    const HistReduce *red_d = (const HistReduce *)(plan + o_r);


    // the tree driver zeroes these counters per tree and reads them once
    unsigned long long *upd = nullptr;
    if (stats) GBT_TRY(scratch_t(c, kScrUpd, kUpdWords, &upd));

    HistLaunch hl{hp.kind, groups_d, G, hp.max_groups_bins, work_d, nullptr, (int32_t)work.size(), red_d,
                  nullptr, (int32_t)red.size(), (int64_t *)partials};
    hl.timed = ws == nullptr;
    GBT_CHECK(n_sub == 0 || parent_hist, "subtraction needs the parent histograms");
    GBT_TRY(hist_launch_device(c, mx, page, q, rows, hl, parent_hist, hist, upd));
    if (stats && !work.empty()) {
        // algorithmic bytes: the packed symbols of each row, its 16-byte
        // fixed-point pair, its 4-byte row id (when indirect), and one write
        // of every built node's histogram
        int64_t wbytes = 4 * (((int64_t)mx->stride * mx->w + 31) / 32);
        stats->hist_launches += 1;
        stats->hist_rows += total_rows;
        stats->hist_bytes += total_rows * (wbytes + 16 + (rows ? 4 : 0)) + (int64_t)n_build * tb * 16;
    }
    return GBT_OK;
}

constexpr int kMaxDevices = 64;
static std::mutex g_static_mu;
static void *g_static_at[kMaxDevices];  // the static scratch's address on each device

gbt_status static_scratch_init(int device)
{
    if (device < 0 || device >= kMaxDevices)
        return set_error(GBT_E_UNSUPPORTED, "device %d: the static scratch table holds %d devices", device,
                         kMaxDevices);
    std::lock_guard<std::mutex> lk(g_static_mu);
    if (g_static_at[device]) return GBT_OK;
    void *p = nullptr;
    GBT_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(::scratch)));
    if (!p) return set_error(GBT_E_DEVICE, "no device address for the static scratch on device %d", device);
    g_static_at[device] = p;
    return GBT_OK;
}

static gbt_status static_scratch(int device, HistWorkspace *ws)
{
    std::lock_guard<std::mutex> lk(g_static_mu);
    if (device < 0 || device >= kMaxDevices || !g_static_at[device])
        return set_error(GBT_E_INVALID, "no static scratch on device %d (the context did not resolve it)", device);
    ws->base = (char *)g_static_at[device];
    ws->bytes = kStaticScratchBytes;
    return GBT_OK;
}

// A histogram kernel launch on the context stream; with a timer mark the
// launch fills the mark's events with its own start and end (the kernel's
// time, without the dispatch around it).
#define GBT_HIST_LAUNCH(KFN, GRID, BLOCK, LDS, ...)                                                       \
    do {                                                                                                 \
        if (mark >= 0) {                                                                                 \
            hipEvent_t ev_a, ev_b;                                                                       \
            timer_events(c, mark, &ev_a, &ev_b);                                                         \
            hipExtLaunchKernelGGL(KFN, dim3(GRID), dim3(BLOCK), (uint32_t)(LDS), c->stream, ev_a, ev_b, 0u, \
                                  __VA_ARGS__);                                                          \
        } else {                                                                                         \
            KFN<<<GRID, BLOCK, LDS, c->stream>>>(__VA_ARGS__);                                           \
        }                                                                                                \
    } while (0)

gbt_status hist_launch_device(gbt_ctx *c, const gbt_matrix *mx, const uint32_t *page, const int64_t *q,
                              const int32_t *rows, const HistLaunch &hl, const int64_t *parent_hist,
                              int64_t *hist, unsigned long long *upd)
{
    const int64_t tb = mx->total_bins;
    const int32_t G = hl.n_groups;
    longlong2 *partials = (longlong2 *)hl.partials;
    if (!mx->sparse && (mx->w < 1 || mx->w > 12))
        return set_error(GBT_E_UNSUPPORTED, "dense symbols of %d bits", mx->w);
    if (hl.cols.p)
        GBT_CHECK(!rows && !mx->sparse && hl.kind == kHistDense && (hl.cols.bytes == 1 || hl.cols.bytes == 2),
                  "a column copy from a histogram pass needs the plain dense kernel over the page in row order");
    if (hl.max_work > 0 && hl.kind == kHistRot) {
        const uint32_t null_sym = mx->has_missing ? mx->null_sym : 0xffffffffu;
        const unsigned grid = (unsigned)((size_t)hl.max_work * (size_t)G);
        const size_t lds = (size_t)kRotBins * kRotCols * 16;
        const longlong2 *qq = (const longlong2 *)q;
        const int mark = hl.timed ? timer_begin_launch(c, kPhHist) : -1;
#define GBT_HIST_ROT(WB)                                                                                 \
    case WB: {                                                                                           \
        auto kfn = rows ? k_hist_rot<WB, true> : k_hist_rot<WB, false>;                                   \
        GBT_HIST_LAUNCH(kfn, grid, kRotThreads, lds, page, mx->row_words, null_sym, qq, rows, hl.work,     \
                        hl.groups, G, hl.n_work_d, mx->bin_ptr_d, tb, partials, upd);                    \
        break;                                                                                           \
    }
        switch (mx->w) {
            GBT_HIST_ROT(1)
            GBT_HIST_ROT(2)
            GBT_HIST_ROT(3)
            GBT_HIST_ROT(4)
            GBT_HIST_ROT(5)
            GBT_HIST_ROT(6)
            GBT_HIST_ROT(7)
            GBT_HIST_ROT(8)
            GBT_HIST_ROT(9)
            default:
                return set_error(GBT_E_UNSUPPORTED, "rotated histogram kernel with %d-bit symbols", mx->w);
        }
#undef GBT_HIST_ROT
        GBT_LAUNCHED();
    } else if (hl.max_work > 0) {
        uint32_t null_sym = (mx->sparse || mx->has_missing) ? mx->null_sym : 0xffffffffu;
        uint32_t mask = mx->w >= 32 ? 0xffffffffu : ((1u << mx->w) - 1u);
        unsigned grid = (unsigned)((size_t)hl.max_work * (size_t)G);
        const int mark = hl.timed ? timer_begin_launch(c, kPhHist) : -1;
        if (mx->sparse) {
            size_t lds = (size_t)hl.max_groups_bins * 16;
            auto kfn = rows ? k_hist_sparse<true> : k_hist_sparse<false>;
            GBT_HIST_LAUNCH(kfn, grid, kSparseThreads, lds, page, mx->row_words, mx->w, mask, mx->stride,
                            (const longlong2 *)q, rows, hl.work, hl.groups, G, hl.n_work_d, tb, partials, upd,
                            hl.slot_tbl, hl.tbl_stride);
        } else {
            const size_t lds = (size_t)(kDenseBins + hl.max_groups_bins) * 8;
            const longlong2 *qq = (const longlong2 *)q;
#define GBT_HIST_DENSE(WB)                                                                                  \
    case WB: {                                                                                              \
        auto kfn = rows ? k_hist_dense<WB, true> : k_hist_dense<WB, false>;                                  \
        GBT_HIST_LAUNCH(kfn, grid, kHistThreads, lds, page, mx->row_words, null_sym, qq, rows, hl.work,       \
                        hl.groups, G, hl.n_work_d, mx->bin_ptr_d, tb, partials, upd, hl.cols);             \
        break;                                                                                              \
    }
            switch (mx->w) {
                GBT_HIST_DENSE(1)
                GBT_HIST_DENSE(2)
                GBT_HIST_DENSE(3)
                GBT_HIST_DENSE(4)
                GBT_HIST_DENSE(5)
                GBT_HIST_DENSE(6)
                GBT_HIST_DENSE(7)
                GBT_HIST_DENSE(8)
                GBT_HIST_DENSE(9)
                GBT_HIST_DENSE(10)
                GBT_HIST_DENSE(11)
                GBT_HIST_DENSE(12)
            }
#undef GBT_HIST_DENSE
        }
        GBT_LAUNCHED();
    }
    if (hl.max_red > 0) {
        const int aux = hl.timed ? timer_begin(c, kPhHistAux) : -1;
        dim3 rg((unsigned)((tb + kRedBins - 1) / kRedBins), (unsigned)hl.max_red);
        k_hist_reduce<<<rg, kRedBins * kRedSplit, 0, c->stream>>>(partials, hl.red, hl.n_red_d,
                                                                  (const longlong2 *)parent_hist,
                                                                  (longlong2 *)hist, tb);
        GBT_LAUNCHED();
        timer_end(c, aux);
    }
    return GBT_OK;
}

}  // namespace gbt

using namespace gbt;

extern "C" gbt_status gbt_build_hist(gbt_ctx *c, const gbt_matrix *layout, const uint32_t *page_d,
                                     const int64_t *gpair_fx_d, const int32_t *rows_d,
                                     const gbt_seg *build_h, int32_t n_build, const gbt_sub *sub_h,
                                     int32_t n_sub, const int64_t *parent_hist_d, int64_t *hist_d)
{
    GBT_CHECK(c && layout && hist_d, "gbt_build_hist: NULL argument");
    GBT_CHECK(n_build >= 0 && n_sub >= 0, "negative counts");
    GBT_CHECK(n_build == 0 || (page_d && gpair_fx_d && build_h), "gbt_build_hist: NULL rows input");
    GBT_CHECK(n_sub == 0 || (sub_h && parent_hist_d), "gbt_build_hist: NULL subtraction input");
    GBT_CHECK(((uintptr_t)page_d & 15) == 0, "gbt_build_hist: the page must be 16-byte aligned");
    for (int32_t k = 0; k < n_build; ++k)
        GBT_CHECK(build_h[k].begin >= 0 && build_h[k].begin <= build_h[k].end && build_h[k].node_slot >= 0,
                  "bad build segment %d", k);
    GBT_TRY(set_device(c));
    GBT_TRY(build_hist_impl(c, layout, page_d, gpair_fx_d, rows_d, build_h, n_build, sub_h, n_sub,
                            parent_hist_d, hist_d, nullptr));
    GBT_HIP(hipStreamSynchronize(c->stream));
    return GBT_OK;
}

extern "C" gbt_status gbt_build_hist_noalloc(gbt_ctx *c, const gbt_matrix *layout, const uint32_t *page_d,
                                             const int64_t *gpair_fx_d, const int32_t *rows_d,
                                             const gbt_seg *build_h, int32_t n_build, const gbt_sub *sub_h,
                                             int32_t n_sub, const int64_t *parent_hist_d, int64_t *hist_d)
{
    GBT_CHECK(c && layout && hist_d, "gbt_build_hist_noalloc: NULL argument");
    GBT_CHECK(n_build >= 0 && n_sub >= 0, "negative counts");
    GBT_CHECK(n_build == 0 || (page_d && gpair_fx_d && build_h), "gbt_build_hist_noalloc: NULL rows input");
    GBT_CHECK(n_sub == 0 || (sub_h && parent_hist_d), "gbt_build_hist_noalloc: NULL subtraction input");
    GBT_CHECK(((uintptr_t)page_d & 15) == 0, "gbt_build_hist_noalloc: the page must be 16-byte aligned");
    for (int32_t k = 0; k < n_build; ++k)
        GBT_CHECK(build_h[k].begin >= 0 && build_h[k].begin <= build_h[k].end && build_h[k].node_slot >= 0,
                  "bad build segment %d", k);
    GBT_TRY(set_device(c));
    HistWorkspace ws;
    GBT_TRY(static_scratch(c->device, &ws));
    GBT_TRY(build_hist_impl(c, layout, page_d, gpair_fx_d, rows_d, build_h, n_build, sub_h, n_sub,
                            parent_hist_d, hist_d, nullptr, &ws));
    GBT_HIP(hipStreamSynchronize(c->stream));
    return GBT_OK;
}
