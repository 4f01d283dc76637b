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

#include <algorithm>
#include <cstring>

namespace gbt {

constexpr int kHistThreads = 512;
constexpr int kLdsBins = 4096;  // 64 KiB of int64 (g, h) per workgroup

// A dense group spans at most this many words of a row and this many features.
constexpr int kGroupWords = 8;
constexpr int kMaxGroupFeat = 32;

// Zero the LDS histogram (sg | sh, nb bins each).
__device__ inline void lds_zero(unsigned long long *lds, int32_t nb)
{
    for (int t = threadIdx.x; t < 2 * nb; t += kHistThreads) lds[t] = 0ull;
    __syncthreads();
}

// Write the LDS histogram as the chunk's partial and count the updates.
__device__ inline void lds_flush(const unsigned long long *sg, const unsigned long long *sh,
                                 int32_t nb, longlong2 *__restrict__ dst, unsigned int cnt,
                                 unsigned long long *__restrict__ n_updates)
{
    __syncthreads();
    for (int t = threadIdx.x; t < nb; t += kHistThreads)
        dst[t] = make_longlong2((long long)sg[t], (long long)sh[t]);
    if (n_updates) {
        // one atomic per block, spread over kUpdCounters addresses
        __shared__ unsigned int red[kHistThreads / 64];
        for (int d = 32; d > 0; d >>= 1) cnt += __shfl_xor(cnt, d, 64);
        if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = cnt;
        __syncthreads();
        if (threadIdx.x == 0) {
            unsigned long long t = 0;
            for (int w = 0; w < kHistThreads / 64; ++w) t += red[w];
            if (t) atomicAdd(&n_updates[blockIdx.x % kUpdCounters], t);
        }
    }
}

// Dense rows: slot j holds feature j.  The group's bin offsets live in scalar
// registers; each lane fetches the next row's pair and words while it
// decodes the current row from a register queue (constant indices only).
template <bool kRows>
__global__ void __launch_bounds__(kHistThreads)
    k_hist_dense(const uint32_t *__restrict__ page, int32_t row_words, int32_t w, uint32_t mask,
                 uint32_t null_sym, const longlong2 *__restrict__ q, const int32_t *__restrict__ rows,
                 const HistWork *__restrict__ work, const HistGroup *__restrict__ groups,
                 int32_t n_groups, const int32_t *__restrict__ n_work_d, const int32_t *__restrict__ bin_ptr,
                 int64_t total_bins, longlong2 *__restrict__ partials,
                 unsigned long long *__restrict__ n_updates)
{
    extern __shared__ unsigned long long lds[];
    const uint32_t active = n_work_d ? (uint32_t)(*n_work_d * n_groups) : gridDim.x;
    if (blockIdx.x >= active) return;
    const uint32_t L = xcd_remap(blockIdx.x, active);
    const HistWork wk = work[L / n_groups];
    const HistGroup gr = groups[L % n_groups];
    const int32_t nb = gr.b1 - gr.b0, nf = gr.f1 - gr.f0;
    unsigned long long *sg = lds, *sh = lds + nb;
    int32_t off[kMaxGroupFeat];
#pragma unroll
    for (int u = 0; u < kMaxGroupFeat; ++u) off[u] = u < nf ? bin_ptr[gr.f0 + u] - gr.b0 : 0;
    lds_zero(lds, nb);

    unsigned int cnt = 0;
    int64_t i = wk.begin + threadIdx.x;
    longlong2 qn = make_longlong2(0, 0);
    uint32_t wn[kGroupWords];
    auto fetch = [&](int64_t ii) {
        const int64_t r = kRows ? (int64_t)rows[ii] : ii;
        qn = q[r];
        const uint32_t *p = page + r * row_words + gr.w0;
#pragma unroll
        for (int k = 0; k < kGroupWords; ++k) wn[k] = k < gr.nw ? p[k] : 0u;
    };
    if (i < wk.end) fetch(i);
    for (; i < wk.end; i += kHistThreads) {
        const unsigned long long qg = (unsigned long long)qn.x, qh = (unsigned long long)qn.y;
        uint32_t wq[kGroupWords];
#pragma unroll
        for (int k = 0; k < kGroupWords; ++k) wq[k] = wn[k];
        if (i + kHistThreads < wk.end) fetch(i + kHistThreads);
        uint64_t buf = (uint64_t)wq[0] >> gr.skip;
        int32_t nbits = 32 - gr.skip;
#pragma unroll
        for (int k = 0; k + 1 < kGroupWords; ++k) wq[k] = wq[k + 1];
#pragma unroll
        for (int u = 0; u < kMaxGroupFeat; ++u) {
            if (u < nf) {
                if (nbits < w) {
                    buf |= (uint64_t)wq[0] << nbits;
                    nbits += 32;
#pragma unroll
                    for (int k = 0; k + 1 < kGroupWords; ++k) wq[k] = wq[k + 1];
                }
                const uint32_t sym = (uint32_t)buf & mask;
                buf >>= w;
                nbits -= w;
                if (sym != null_sym) {
                    const int32_t idx = off[u] + (int32_t)sym;
                    atomicAdd(&sg[idx], qg);
                    atomicAdd(&sh[idx], qh);
                    ++cnt;
                }
            }
        }
    }
    lds_flush(sg, sh, nb, partials + (int64_t)wk.part * total_bins + gr.b0, cnt, n_updates);
}

// Sparse rows: the row's present features in ascending order as global
// bins, null padded; the group keeps the symbols in its bin range.
template <bool kRows>
__global__ void __launch_bounds__(kHistThreads)
    k_hist_sparse(const uint32_t *__restrict__ page, int32_t row_words, int32_t w, uint32_t mask,
                  int32_t stride, const longlong2 *__restrict__ q, const int32_t *__restrict__ rows,
                  const HistWork *__restrict__ work, const HistGroup *__restrict__ groups,
                  int32_t n_groups, const int32_t *__restrict__ n_work_d, int64_t total_bins,
                  longlong2 *__restrict__ partials, unsigned long long *__restrict__ n_updates)
{
    extern __shared__ unsigned long long lds[];
    const uint32_t active = n_work_d ? (uint32_t)(*n_work_d * n_groups) : gridDim.x;
    if (blockIdx.x >= active) return;
    const uint32_t L = xcd_remap(blockIdx.x, active);
    const HistWork wk = work[L / n_groups];
    const HistGroup gr = groups[L % n_groups];
    const int32_t nb = gr.b1 - gr.b0;
    unsigned long long *sg = lds, *sh = lds + nb;
    lds_zero(lds, nb);
    unsigned int cnt = 0;
    for (int64_t i = wk.begin + threadIdx.x; i < wk.end; i += kHistThreads) {
        const int64_t r = kRows ? (int64_t)rows[i] : i;
        const longlong2 qq = q[r];
        const unsigned long long qg = (unsigned long long)qq.x, qh = (unsigned long long)qq.y;
        const uint32_t *p = page + r * row_words;
        uint64_t buf = (uint64_t)(*p++);
        int32_t nbits = 32;
        for (int32_t s = 0; s < stride; ++s) {
            if (nbits < w) {
                buf |= (uint64_t)(*p++) << nbits;
                nbits += 32;
            }
            const uint32_t sym = (uint32_t)buf & mask;
            buf >>= w;
            nbits -= w;
            if (sym >= (uint32_t)gr.b1) break;  // ascending; padding is the largest symbol
            if (sym >= (uint32_t)gr.b0) {
                const int32_t idx = (int32_t)sym - gr.b0;
                atomicAdd(&sg[idx], qg);
                atomicAdd(&sh[idx], qh);
                ++cnt;
            }
        }
    }
    lds_flush(sg, sh, nb, partials + (int64_t)wk.part * total_bins + gr.b0, cnt, n_updates);
}

__global__ void k_hist_reduce(const longlong2 *__restrict__ partials, const HistReduce *__restrict__ red,
                              const int32_t *__restrict__ n_red_d, const longlong2 *__restrict__ parent,
                              longlong2 *__restrict__ hist, int64_t total_bins)
{
    if (n_red_d && (int32_t)blockIdx.y >= *n_red_d) return;
    const HistReduce rd = red[blockIdx.y];
    for (int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; b < total_bins;
         b += (int64_t)gridDim.x * blockDim.x) {
        long long g = 0, h = 0;
        for (int32_t k = 0; k < rd.nparts; ++k) {
            longlong2 v = partials[(int64_t)(rd.part0 + k) * total_bins + b];
            g += v.x;
            h += v.y;
        }
        hist[(int64_t)rd.slot * total_bins + b] = make_longlong2(g, h);
        if (rd.sub_target >= 0) {
            longlong2 pv = parent[(int64_t)rd.sub_parent * total_bins + b];
            hist[(int64_t)rd.sub_target * total_bins + b] = make_longlong2(pv.x - g, pv.y - h);
        }
    }
}

// Feature groups with at most kLdsBins bins each and about equal bin counts;
// a dense group's symbols also span at most kGroupWords words.
bool hist_groups(const gbt_matrix *mx, std::vector<HistGroup> *out)
{
    out->clear();
    bool fits = true;
    const int64_t tb = mx->total_bins;
    const int64_t G = std::max<int64_t>(1, (tb + kLdsBins - 1) / kLdsBins);
    const int64_t target = (tb + G - 1) / G;
    auto span_words = [&](int32_t f0, int32_t f1) {
        int64_t b0 = (int64_t)f0 * mx->w, b1 = (int64_t)f1 * mx->w;
        return (int32_t)((b1 + 31) / 32 - b0 / 32);
    };
    int32_t f0 = 0;
    while (f0 < mx->m) {
        int32_t f1 = f0 + 1;
        while (f1 < mx->m && mx->bin_ptr_h[f1 + 1] - mx->bin_ptr_h[f0] <= target &&
               (mx->sparse || (span_words(f0, f1 + 1) <= kGroupWords && f1 + 1 - f0 <= kMaxGroupFeat)))
            ++f1;
        HistGroup g;
        g.f0 = f0;
        g.f1 = f1;
        g.b0 = mx->bin_ptr_h[f0];
        g.b1 = mx->bin_ptr_h[f1];
        int64_t bit = (int64_t)f0 * mx->w;
        g.w0 = (int32_t)(bit >> 5);
        g.skip = (int32_t)(bit & 31);
        g.nw = span_words(f0, f1);
        g.pad0 = 0;
        if (g.b1 - g.b0 > kLdsBins) fits = false;
        if (!mx->sparse && g.nw > kGroupWords) fits = false;
        out->push_back(g);
        f0 = f1;
    }
    return fits;
}

gbt_status build_hist_impl(gbt_ctx *c, const gbt_matrix *mx, const uint32_t *page, const int64_t *q,
                           const int32_t *rows, const gbt_seg *build, int32_t n_build,
                           const gbt_sub *sub, int32_t n_sub, const int64_t *parent_hist,
                           int64_t *hist, gbt_tree_stats *stats)
{
    const int64_t tb = mx->total_bins;
    if (tb == 0 || n_build == 0) {
        GBT_CHECK(n_sub == 0, "a subtraction needs its built sibling in the same call");
        return GBT_OK;
    }
    std::vector<HistGroup> groups;
    const bool fits = hist_groups(mx, &groups);
    if (!fits)
        return set_error(GBT_E_UNSUPPORTED, "a feature has more than %d bins or %d words of symbols",
                         kLdsBins, kGroupWords);
    const int32_t G = (int32_t)groups.size();

    int64_t total_rows = 0;
    for (int32_t k = 0; k < n_build; ++k) total_rows += std::max<int64_t>(0, build[k].end - build[k].begin);
    // chunks: about two workgroups per CU over all groups, at least 2048 rows each
    const int64_t target_wg = 2 * kCUs;
    int64_t chunk = (total_rows * G + target_wg - 1) / target_wg;
    chunk = std::max<int64_t>(chunk, 2048);
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
    size_t o_w = ((size_t)G * sizeof(HistGroup) + 255) / 256 * 256;
    size_t o_r = o_w + (std::max<size_t>(work.size(), 1) * sizeof(HistWork) + 255) / 256 * 256;
    size_t bytes = o_r + red.size() * sizeof(HistReduce) + 256;
    char *plan;
    GBT_TRY(scratch_t(c, kScrWork, bytes, &plan));
    std::vector<char> h(bytes);
    memcpy(h.data(), groups.data(), G * sizeof(HistGroup));
    if (!work.empty()) memcpy(h.data() + o_w, work.data(), work.size() * sizeof(HistWork));
    memcpy(h.data() + o_r, red.data(), red.size() * sizeof(HistReduce));
    GBT_HIP(hipMemcpyAsync(plan, h.data(), bytes, hipMemcpyHostToDevice, c->stream));
    const HistGroup *groups_d = (const HistGroup *)plan;
    const HistWork *work_d = (const HistWork *)(plan + o_w);
    const HistReduce *red_d = (const HistReduce *)(plan + o_r);

    longlong2 *partials = nullptr;
    GBT_TRY(scratch(c, kScrPartials, (size_t)std::max(nparts, 1) * tb * 16, (void **)&partials));

    // the tree driver zeroes these counters per tree and reads them once
    unsigned long long *upd = nullptr;
    if (stats) GBT_TRY(scratch_t(c, kScrUpd, kUpdCounters, &upd));

    HistLaunch hl{groups_d, G, 0, work_d, nullptr, (int32_t)work.size(), red_d, nullptr, (int32_t)red.size(),
                  (int64_t *)partials};
    for (auto &g : groups) hl.max_groups_bins = std::max(hl.max_groups_bins, g.b1 - g.b0);
    GBT_CHECK(n_sub == 0 || parent_hist, "subtraction needs the parent histograms");
    GBT_TRY(hist_launch_device(c, mx, page, q, rows, hl, parent_hist, hist, upd));
    if (stats && !work.empty()) {
        // algorithmic bytes: the packed symbols of each row, its 16-byte
        // fixed-point pair, its 4-byte row id (when indirect), and one write
        // of every chunk's partial histogram
        int64_t wbytes = 4 * (((int64_t)mx->stride * mx->w + 31) / 32);
        stats->hist_launches += 1;
        stats->hist_rows += total_rows;
        stats->hist_bytes += total_rows * (wbytes + 16 + (rows ? 4 : 0)) + (int64_t)nparts * tb * 16;
    }
    return GBT_OK;
}

gbt_status hist_launch_device(gbt_ctx *c, const gbt_matrix *mx, const uint32_t *page, const int64_t *q,
                              const int32_t *rows, const HistLaunch &hl, const int64_t *parent_hist,
                              int64_t *hist, unsigned long long *upd)
{
    const int64_t tb = mx->total_bins;
    const int32_t G = hl.n_groups;
    longlong2 *partials = (longlong2 *)hl.partials;
    if (hl.max_work > 0) {
        size_t lds = (size_t)hl.max_groups_bins * 16;
        uint32_t null_sym = (mx->sparse || mx->has_missing) ? mx->null_sym : 0xffffffffu;
        uint32_t mask = mx->w >= 32 ? 0xffffffffu : ((1u << mx->w) - 1u);
        unsigned grid = (unsigned)((size_t)hl.max_work * (size_t)G);
        const int mark = timer_begin(c, kPhHist);
#define GBT_HIST_DENSE(RW)                                                                          \
    k_hist_dense<RW><<<grid, kHistThreads, lds, c->stream>>>(page, mx->row_words, mx->w, mask, null_sym,   \
                                                             (const longlong2 *)q, rows, hl.work,        \
                                                             hl.groups, G, hl.n_work_d, mx->bin_ptr_d, tb, \
                                                             partials, upd)
#define GBT_HIST_SPARSE(RW)                                                                        \
    k_hist_sparse<RW><<<grid, kHistThreads, lds, c->stream>>>(page, mx->row_words, mx->w, mask,      \
                                                              mx->stride, (const longlong2 *)q, rows,  \
                                                              hl.work, hl.groups, G, hl.n_work_d, tb,  \
                                                              partials, upd)
        if (mx->sparse) {
            if (rows)
                GBT_HIST_SPARSE(true);
            else
                GBT_HIST_SPARSE(false);
        } else {
            if (rows)
                GBT_HIST_DENSE(true);
            else
                GBT_HIST_DENSE(false);
        }
#undef GBT_HIST_DENSE
#undef GBT_HIST_SPARSE
        GBT_LAUNCHED();
        timer_end(c, mark);
    }
    if (hl.max_red > 0) {
        const int aux = timer_begin(c, kPhHistAux);
        dim3 rg((unsigned)std::min<int64_t>((tb + 255) / 256, 256), (unsigned)hl.max_red);
        k_hist_reduce<<<rg, 256, 0, c->stream>>>(partials, hl.red, hl.n_red_d, (const longlong2 *)parent_hist,
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
    for (int32_t k = 0; k < n_build; ++k)
        GBT_CHECK(build_h[k].begin >= 0 && build_h[k].begin <= build_h[k].end && build_h[k].node_slot >= 0,
                  "bad build segment %d", k);
    GBT_TRY(set_device(c));
    GBT_TRY(build_hist_impl(c, layout, page_d, gpair_fx_d, rows_d, build_h, n_build, sub_h, n_sub,
                            parent_hist_d, hist_d, nullptr));
    GBT_HIP(hipStreamSynchronize(c->stream));
    return GBT_OK;
}
