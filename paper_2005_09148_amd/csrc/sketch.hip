// sketch.hip -- Sec. 3.1 / Alg. 3 on the device: a batch's sample keys,
// sorted per feature (a segmented LSD radix sort), become per-feature
// summaries that are merged into the running summary (sketch_impl.h gives
// the rules).  Every feature is independent: one segment, one block.
#include "sketch_impl.h"
#include "wave_impl.h"

#include <algorithm>
#include <cstring>

namespace gbt {

namespace {

constexpr uint32_t kNanKey = 0xffffffffu;

// ------------------------------------------------------------ radix sort
// Keys of one segment are cut into tiles of kSortTile; a pass sorts by one
// 8-bit digit: per-tile digit counts, their offsets per segment (digits in
// order, tiles in order within a digit), then a stable scatter of each tile
// (the tile is first sorted by the digit in LDS with eight stable one-bit
// splits).  Four passes sort 32-bit keys.
constexpr int kSortThreads = 256;
constexpr int kSortItems = 16;
constexpr int kSortTile = kSortThreads * kSortItems;
constexpr int kSortPad = kSortTile + kSortTile / kSortItems;  // one word of padding per 16

struct SortTile {
    int64_t begin;  // first key of the tile
    int64_t seg0;   // first key of its segment
    int32_t len;    // keys in the tile (<= kSortTile)
    int32_t seg;
};

__device__ inline int pad_idx(int i) { return i + i / kSortItems; }

__global__ void __launch_bounds__(kSortThreads)
    k_sort_hist(const uint32_t *__restrict__ in, const SortTile *__restrict__ tiles, int32_t shift,
                uint32_t *__restrict__ hist)
{
    __shared__ uint32_t cnt[256];
    cnt[threadIdx.x] = 0;
    __syncthreads();
    const SortTile t = tiles[blockIdx.x];
    for (int32_t i = threadIdx.x; i < t.len; i += kSortThreads) atomicAdd(&cnt[(in[t.begin + i] >> shift) & 255u], 1u);
    __syncthreads();
    hist[(int64_t)blockIdx.x * 256 + threadIdx.x] = cnt[threadIdx.x];
}

// One block per segment, a thread per digit: the tiles' counts become the
// position (within the segment) of each tile's first key of each digit.
__global__ void __launch_bounds__(256)
    k_sort_offsets(uint32_t *__restrict__ hist, const int32_t *__restrict__ seg_tiles,
                   const SortTile *__restrict__ tiles)
{
    __shared__ uint32_t wsum[4];
    const int32_t t0 = seg_tiles[blockIdx.x], t1 = seg_tiles[blockIdx.x + 1];
    if (t0 == t1) return;
    const int d = threadIdx.x, lane = d & 63, wid = d >> 6;
    uint32_t total = 0;
    for (int32_t t = t0; t < t1; ++t) total += hist[(int64_t)t * 256 + d];
    const uint32_t x = wave_incl_sum(total);
    if (lane == 63) wsum[wid] = x;
    __syncthreads();
    uint32_t base = x - total;
    for (int w = 0; w < wid; ++w) base += wsum[w];
    uint32_t off = base;
    for (int32_t t = t0; t < t1; ++t) {
        const uint32_t c = hist[(int64_t)t * 256 + d];
        hist[(int64_t)t * 256 + d] = off;
        off += c;
    }
}

// Exclusive scan of v over the 256 threads; *total receives the sum.
__device__ inline int32_t sort_block_scan(int32_t v, int32_t *wsum, int32_t *total)
{
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    const int32_t x = wave_incl_sum(v);
    __syncthreads();
    if (lane == 63) wsum[wid] = x;
    __syncthreads();
    int32_t off = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < kSortThreads / 64; ++w) {
        off += w < wid ? wsum[w] : 0;
        tot += wsum[w];
    }
    *total = tot;
    return x - v + off;
}

__global__ void __launch_bounds__(kSortThreads)
    k_sort_scatter(const uint32_t *__restrict__ in, uint32_t *__restrict__ out, const SortTile *__restrict__ tiles,
                   int32_t shift, const uint32_t *__restrict__ hist)
{
    __shared__ uint32_t sk[kSortPad];
    __shared__ int32_t wsum[kSortThreads / 64];
    __shared__ uint32_t dcnt[256];
    const SortTile t = tiles[blockIdx.x];
    // coalesced loads into LDS; keys past the tile are the largest key and
    // sort (stably) after every real key
    for (int i = threadIdx.x; i < kSortTile; i += kSortThreads) sk[pad_idx(i)] = i < t.len ? in[t.begin + i] : kNanKey;
    dcnt[threadIdx.x] = 0;
    __syncthreads();
    const int base = threadIdx.x * kSortItems;
    uint32_t k[kSortItems];
#pragma unroll
    for (int j = 0; j < kSortItems; ++j) k[j] = sk[pad_idx(base + j)];
    // eight stable splits by the digit's bits, low to high
    for (int r = 0; r < 8; ++r) {
        int32_t zeros = 0;
#pragma unroll
        for (int j = 0; j < kSortItems; ++j) zeros += ((k[j] >> (shift + r)) & 1u) ? 0 : 1;
        int32_t Z;
        const int32_t zb = sort_block_scan(zeros, wsum, &Z);
        int32_t zi = zb, oi = Z + (base - zb);
        __syncthreads();  // every thread has read its keys
#pragma unroll
        for (int j = 0; j < kSortItems; ++j) {
            const bool one = (k[j] >> (shift + r)) & 1u;
            sk[pad_idx(one ? oi++ : zi++)] = k[j];
        }
        __syncthreads();
#pragma unroll
        for (int j = 0; j < kSortItems; ++j) k[j] = sk[pad_idx(base + j)];
    }
    // each digit's first position in the sorted tile
#pragma unroll
    for (int j = 0; j < kSortItems; ++j)
        if (base + j < t.len) atomicAdd(&dcnt[(k[j] >> shift) & 255u], 1u);
    __syncthreads();
    int32_t tot;
    const int32_t dstart = sort_block_scan((int32_t)dcnt[threadIdx.x], wsum, &tot);
    __syncthreads();
    dcnt[threadIdx.x] = (uint32_t)dstart;
    __syncthreads();
    const uint32_t *ho = hist + (int64_t)blockIdx.x * 256;
#pragma unroll
    for (int j = 0; j < kSortItems; ++j) {
        const int p = base + j;
        if (p < t.len) {
            const uint32_t d = (k[j] >> shift) & 255u;
            out[t.seg0 + (int64_t)ho[d] + (p - (int32_t)dcnt[d])] = k[j];
        }
    }
}

// ------------------------------------------------------------ summaries
constexpr int kSumThreads = 1024;

// Exclusive scan across kSumThreads threads; *total receives the sum.
__device__ inline int32_t sum_block_scan(int32_t v, int32_t *wsum, int32_t *total)
{
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    const int32_t x = wave_incl_sum(v);
    __syncthreads();
    if (lane == 63) wsum[wid] = x;
    __syncthreads();
    int32_t off = 0, tot = 0;
    for (int w = 0; w < kSumThreads / 64; ++w) {
        off += w < wid ? wsum[w] : 0;
        tot += wsum[w];
    }
    *total = tot;
    return x - v + off;
}

__device__ inline int64_t block_sum64(int64_t v, long long *wsum)
{
    v = wave_total(v);
    __syncthreads();
    if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = v;
    __syncthreads();
    int64_t t = 0;
    for (int w = 0; w < kSumThreads / 64; ++w) t += wsum[w];
    return t;
}

// first index in [0, n) with a[i] >= x (n if none)
__device__ inline int64_t lower_bound_u32(const uint32_t *a, int64_t n, uint32_t x)
{
    int64_t lo = 0, hi = n;
    while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if (a[mid] < x)
            lo = mid + 1;
        else
            hi = mid;
    }
    return lo;
}

// first index in [0, n) with a[i] > x
__device__ inline int64_t upper_bound_u32(const uint32_t *a, int64_t n, uint32_t x)
{
    int64_t lo = 0, hi = n;
    while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if (a[mid] <= x)
            lo = mid + 1;
        else
            hi = mid;
    }
    return lo;
}

// first index in [0, n) with c[i] >= x
__device__ inline int64_t lower_bound_i64(const long long *c, int64_t n, long long x)
{
    int64_t lo = 0, hi = n;
    while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if (c[mid] < x)
            lo = mid + 1;
        else
            hi = mid;
    }
    return lo;
}

// The summary of one batch, one block per feature: the feature's sorted
// keys a[0, len), missing (NaN) keys last.  When the batch has at most S
// distinct values, all of them with their counts; else the values at ranks
// ceil(tN/S), t = 1..S, each once.
__global__ void __launch_bounds__(kSumThreads)
    k_batch_summary(const uint32_t *__restrict__ keys, const int64_t *__restrict__ seg_begin,
                    const int64_t *__restrict__ seg_len, int32_t S, uint32_t *__restrict__ ov,
                    long long *__restrict__ oc, int64_t *__restrict__ ok)
{
    __shared__ int32_t wsum[kSumThreads / 64];
    __shared__ long long wsum64[kSumThreads / 64];
    __shared__ int64_t s_n;
    const int32_t j = blockIdx.x;
    const uint32_t *a = keys + seg_begin[j];
    const int64_t len = seg_len[j];
    if (threadIdx.x == 0) s_n = lower_bound_u32(a, len, kNanKey);  // values that are not missing
    __syncthreads();
    const int64_t N = s_n;
    uint32_t *v = ov + (int64_t)j * S;
    long long *c = oc + (int64_t)j * S;
    // distinct values: the last position of each run of equal keys
    int64_t runs = 0;
    for (int64_t i = threadIdx.x; i < N; i += kSumThreads) runs += (i == N - 1 || a[i] != a[i + 1]) ? 1 : 0;
    const int64_t K = block_sum64(runs, wsum64);
    int64_t written = 0;
    if (K <= S) {
        constexpr int kPer = 8;
        for (int64_t c0 = 0; c0 < N; c0 += (int64_t)kSumThreads * kPer) {
            const int64_t i0 = c0 + (int64_t)threadIdx.x * kPer;
            uint32_t ends = 0;
            int32_t cnt = 0;
#pragma unroll
            for (int q = 0; q < kPer; ++q) {
                const int64_t i = i0 + q;
                if (i < N && (i == N - 1 || a[i] != a[i + 1])) {
                    ends |= 1u << q;
                    ++cnt;
                }
            }
            int32_t tot;
            int32_t o = sum_block_scan(cnt, wsum, &tot);
#pragma unroll
            for (int q = 0; q < kPer; ++q)
                if ((ends >> q) & 1u) {
                    v[written + o] = a[i0 + q];
                    c[written + o] = i0 + q + 1;
                    ++o;
                }
            written += tot;
        }
    } else {
        // entry t: the value at rank ceil(tN/S), kept unless the entry
        // before it has the same value
        for (int32_t t0 = 1; t0 <= S; t0 += kSumThreads) {
            const int32_t t = t0 + (int32_t)threadIdx.x;
            uint32_t x = 0;
            bool keep = false;
            if (t <= S) {
                const int64_t p = ((int64_t)t * N + S - 1) / S - 1;
                x = a[p];
                keep = t == 1 || a[((int64_t)(t - 1) * N + S - 1) / S - 1] != x;
            }
            int32_t tot;
            const int32_t o = sum_block_scan(keep ? 1 : 0, wsum, &tot);
            if (keep) {
                v[written + o] = x;
                c[written + o] = upper_bound_u32(a, N, x);
            }
            written += tot;
        }
    }
    if (threadIdx.x == 0) ok[j] = written;
}

// Running summary R (k_r entries) merged with the batch summary B, pruned to
// S entries, into O; one block per feature.  U is room for 2S entries and P
// for S counters.  A value's place in the union is the number of distinct
// values below it: those of A, plus those of B, less the ones both hold.
__global__ void __launch_bounds__(kSumThreads)
    k_summary_merge(const uint32_t *__restrict__ rv, const long long *__restrict__ rc, const int64_t *__restrict__ rk,
                    const uint32_t *__restrict__ bv, const long long *__restrict__ bc, const int64_t *__restrict__ bk,
                    int32_t S, uint32_t *__restrict__ uv, long long *__restrict__ uc, int32_t *__restrict__ pre,
                    uint32_t *__restrict__ ov, long long *__restrict__ oc, int64_t *__restrict__ ok)
{
    __shared__ int32_t wsum[kSumThreads / 64];
    const int32_t j = blockIdx.x;
    const int64_t o_f = (int64_t)j * S;
    const uint32_t *A = rv + o_f, *B = bv + o_f;
    const long long *Ac = rc + o_f, *Bc = bc + o_f;
    const int64_t ka = rk[j], kb = bk[j];
    uint32_t *Uv = uv + 2 * o_f;
    long long *Uc = uc + 2 * o_f;
    int32_t *P = pre + o_f;
    const long long N = (ka ? Ac[ka - 1] : 0) + (kb ? Bc[kb - 1] : 0);
    // P[i]: how many of B[0, i) A holds too
    int32_t common = 0;
    for (int64_t c0 = 0; c0 < kb; c0 += kSumThreads) {
        const int64_t i = c0 + threadIdx.x;
        int32_t in_a = 0;
        if (i < kb) {
            const int64_t lt = lower_bound_u32(A, ka, B[i]);
            in_a = (lt < ka && A[lt] == B[i]) ? 1 : 0;
        }
        int32_t tot;
        const int32_t o = sum_block_scan(in_a, wsum, &tot);
        if (i < kb) P[i] = common + o;
        common += tot;
    }
    __syncthreads();  // P is written
    for (int64_t i = threadIdx.x; i < ka; i += kSumThreads) {
        const uint32_t x = A[i];
        const int64_t lt = lower_bound_u32(B, kb, x);
        const int64_t le = lt + ((lt < kb && B[lt] == x) ? 1 : 0);
        const int64_t pos = i + lt - (lt < kb ? P[lt] : common);
        Uv[pos] = x;
        Uc[pos] = Ac[i] + (le ? Bc[le - 1] : 0);
    }
    for (int64_t i = threadIdx.x; i < kb; i += kSumThreads) {
        const uint32_t x = B[i];
        const int64_t lt = lower_bound_u32(A, ka, x);
        if (lt < ka && A[lt] == x) continue;  // placed with A's entry
        const int64_t pos = lt + i - P[i];
        Uv[pos] = x;
        Uc[pos] = Bc[i] + (lt ? Ac[lt - 1] : 0);
    }
    const int64_t ku = ka + kb - common;
    __syncthreads();  // U is written
    uint32_t *Ov = ov + o_f;
    long long *Oc = oc + o_f;
    int64_t written = 0;
    if (ku <= S) {
        for (int64_t i = threadIdx.x; i < ku; i += kSumThreads) {
            Ov[i] = Uv[i];
            Oc[i] = Uc[i];
        }
        written = ku;
    } else {
        for (int32_t t0 = 1; t0 <= S; t0 += kSumThreads) {
            const int32_t t = t0 + (int32_t)threadIdx.x;
            int64_t it = -1;
            bool keep = false;
            if (t <= S) {
                it = lower_bound_i64(Uc, ku, ((long long)t * N + S - 1) / S);
                keep = t == 1 || lower_bound_i64(Uc, ku, ((long long)(t - 1) * N + S - 1) / S) != it;
            }
            int32_t tot;
            const int32_t o = sum_block_scan(keep ? 1 : 0, wsum, &tot);
            if (keep) {
                Ov[written + o] = Uv[it];
                Oc[written + o] = Uc[it];
            }
            written += tot;
        }
    }
    if (threadIdx.x == 0) ok[j] = written;
}

__global__ void k_zero_i64(int64_t *p, int64_t n)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0;
}

}  // namespace

gbt_status merge_sketch_init(gbt_ctx *c, MergeSketch *ms, int32_t m, int32_t S)
{
    ms->m = m;
    ms->S = S;
    ms->cur = 0;
    auto get = [&](size_t bytes, void **p) -> gbt_status {
        GBT_TRY(dev_alloc(c, std::max<size_t>(bytes, 16), p));
        ms->owned.push_back({*p, std::max<size_t>(bytes, 16)});
        return GBT_OK;
    };
    const size_t e = (size_t)m * (size_t)S;
    for (SummarySet *s : {&ms->run[0], &ms->run[1], &ms->batch}) {
        GBT_TRY(get(e * 4, (void **)&s->v));
        GBT_TRY(get(e * 8, (void **)&s->c));
        GBT_TRY(get((size_t)m * 8, (void **)&s->k));
    }
    GBT_TRY(get(2 * e * 4, (void **)&ms->uv));
    GBT_TRY(get(2 * e * 8, (void **)&ms->uc));
    GBT_TRY(get(e * 4, (void **)&ms->pre));
    k_zero_i64<<<(unsigned)((m + 255) / 256), 256, 0, c->stream>>>(ms->run[0].k, m);
    GBT_LAUNCHED();
    return GBT_OK;
}

void merge_sketch_free(gbt_ctx *c, MergeSketch *ms)
{
    (void)hipStreamSynchronize(c->stream);
    for (auto &p : ms->owned) dev_free(c, p.first, p.second);
    ms->owned.clear();
    if (ms->sort_tmp) dev_free(c, ms->sort_tmp, ms->sort_tmp_bytes);
    ms->sort_tmp = nullptr;
    ms->sort_tmp_bytes = 0;
}

gbt_status merge_sketch_add(gbt_ctx *c, MergeSketch *ms, uint32_t *keys, const int64_t *seg_begin_h,
                            const int64_t *seg_len_h)
{
    const int32_t m = ms->m;
    // tiles of every segment
    std::vector<SortTile> tiles;
    std::vector<int32_t> seg_tiles(m + 1, 0);
    int64_t end = 0;
    for (int32_t j = 0; j < m; ++j) {
        GBT_CHECK(seg_len_h[j] >= 0 && seg_len_h[j] < ((int64_t)1 << 31) && seg_begin_h[j] >= 0,
                  "sketch segment %d of %lld keys", j, (long long)seg_len_h[j]);
        seg_tiles[j] = (int32_t)tiles.size();
        for (int64_t b = 0; b < seg_len_h[j]; b += kSortTile)
            tiles.push_back({seg_begin_h[j] + b, seg_begin_h[j], (int32_t)std::min<int64_t>(kSortTile, seg_len_h[j] - b), j});
        end = std::max(end, seg_begin_h[j] + seg_len_h[j]);
    }
    seg_tiles[m] = (int32_t)tiles.size();
    const int64_t nt = (int64_t)tiles.size();
    GBT_CHECK(nt < INT32_MAX, "sketch batch of %lld sort tiles", (long long)nt);
    // scratch: the second key buffer | tiles | tile starts | histograms | segments
    auto al = [](size_t b) { return (b + 255) / 256 * 256; };
    const size_t o_tiles = al((size_t)end * 4), o_st = o_tiles + al(std::max<int64_t>(nt, 1) * sizeof(SortTile));
    const size_t o_hist = o_st + al((size_t)(m + 1) * 4), o_seg = o_hist + al((size_t)std::max<int64_t>(nt, 1) * 1024);
    const size_t bytes = o_seg + 2 * al((size_t)m * 8);
    if (ms->sort_tmp_bytes < bytes) {
        GBT_HIP(hipStreamSynchronize(c->stream));
        if (ms->sort_tmp) dev_free(c, ms->sort_tmp, ms->sort_tmp_bytes);
        ms->sort_tmp = nullptr;
        ms->sort_tmp_bytes = 0;
        GBT_TRY(dev_alloc(c, bytes, &ms->sort_tmp));
        ms->sort_tmp_bytes = bytes;
    }
    char *base = (char *)ms->sort_tmp;
    uint32_t *alt = (uint32_t *)base;
    SortTile *tiles_d = (SortTile *)(base + o_tiles);
    int32_t *st_d = (int32_t *)(base + o_st);
    uint32_t *hist = (uint32_t *)(base + o_hist);
    int64_t *sb_d = (int64_t *)(base + o_seg), *sl_d = (int64_t *)(base + o_seg + al((size_t)m * 8));
    // one upload of the small tables (then the host arrays may go)
    std::vector<char> h(bytes - o_tiles, 0);
    if (nt) memcpy(h.data(), tiles.data(), (size_t)nt * sizeof(SortTile));
    memcpy(h.data() + (o_st - o_tiles), seg_tiles.data(), (size_t)(m + 1) * 4);
    memcpy(h.data() + (o_seg - o_tiles), seg_begin_h, (size_t)m * 8);
    memcpy(h.data() + (o_seg + al((size_t)m * 8) - o_tiles), seg_len_h, (size_t)m * 8);
    GBT_HIP(hipMemcpyAsync(base + o_tiles, h.data(), h.size(), hipMemcpyHostToDevice, c->stream));
    if (nt) {
        uint32_t *src = keys, *dst = alt;
        for (int pass = 0; pass < 4; ++pass) {
            const int32_t shift = 8 * pass;
            k_sort_hist<<<(unsigned)nt, kSortThreads, 0, c->stream>>>(src, tiles_d, shift, hist);
            GBT_LAUNCHED();
            k_sort_offsets<<<(unsigned)m, 256, 0, c->stream>>>(hist, st_d, tiles_d);
            GBT_LAUNCHED();
            k_sort_scatter<<<(unsigned)nt, kSortThreads, 0, c->stream>>>(src, dst, tiles_d, shift, hist);
            GBT_LAUNCHED();
            std::swap(src, dst);
        }
        // four passes: the sorted keys are back in `keys`
    }
    SummarySet &R = ms->run[ms->cur], &O = ms->run[1 - ms->cur];
    k_batch_summary<<<(unsigned)m, kSumThreads, 0, c->stream>>>(keys, sb_d, sl_d, ms->S, ms->batch.v, ms->batch.c,
                                                                ms->batch.k);
    GBT_LAUNCHED();
    k_summary_merge<<<(unsigned)m, kSumThreads, 0, c->stream>>>(R.v, R.c, R.k, ms->batch.v, ms->batch.c, ms->batch.k,
                                                                ms->S, ms->uv, ms->uc, ms->pre, O.v, O.c, O.k);
    GBT_LAUNCHED();
    ms->cur = 1 - ms->cur;
    // the small tables' host copy must outlive the upload
    GBT_HIP(hipStreamSynchronize(c->stream));
    return GBT_OK;
}

gbt_status merge_sketch_download(gbt_ctx *c, const MergeSketch *ms, std::vector<uint32_t> *v,
                                 std::vector<long long> *cnt, std::vector<int64_t> *k)
{
    const size_t e = (size_t)ms->m * (size_t)ms->S;
    const SummarySet &R = ms->run[ms->cur];
    v->resize(e);
    cnt->resize(e);
    k->resize(ms->m);
    GBT_HIP(hipMemcpyAsync(v->data(), R.v, e * 4, hipMemcpyDeviceToHost, c->stream));
    GBT_HIP(hipMemcpyAsync(cnt->data(), R.c, e * 8, hipMemcpyDeviceToHost, c->stream));
    GBT_HIP(hipMemcpyAsync(k->data(), R.k, (size_t)ms->m * 8, hipMemcpyDeviceToHost, c->stream));
    GBT_HIP(hipStreamSynchronize(c->stream));
    return GBT_OK;
}

}  // namespace gbt
