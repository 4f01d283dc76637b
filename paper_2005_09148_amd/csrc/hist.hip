// hist.hip -- Alg. 1 BuildHistograms on bit-packed ELLPACK rows.
//
// Each workgroup owns one (row chunk of one node, feature group) pair.  A
// feature group is a contiguous feature range whose bins fit the LDS
// budget; its int64 fixed-point (g, h) histogram lives in LDS while the
// chunk's rows stream through (one row per lane, the group's words decoded
// by a running bit buffer), then it is merged into the node's global
// histogram with one 64-bit atomic per non-zero bin.  Work items are mapped
// so that the groups of one chunk run on the same XCD and share its L2 for
// the gradient pairs and row ids.  The sibling of a built child is the
// parent minus the built child, an exact integer subtraction.
#include "common.h"

#include <algorithm>
#include <cstring>

namespace gbt {

constexpr int kHistThreads = 256;
constexpr int kLdsBins = 4096;  // 64 KiB of int64 (g, h) per workgroup

struct HistWork {
    int64_t begin, end;
    int32_t slot;
    int32_t pad0;
};

struct HistGroup {
    int32_t f0, f1;  // features [f0, f1)
    int32_t b0, b1;  // global bins [b0, b1)
    int32_t w0;      // dense: word holding the first bit of feature f0
    int32_t skip;    // dense: bit offset of feature f0 in that word
};

template <bool kSparse, bool kRows>
__global__ void __launch_bounds__(kHistThreads)
    k_hist_lds(const uint32_t *__restrict__ page, int32_t row_words, int32_t w, uint32_t mask,
               uint32_t null_sym, int32_t stride, const longlong2 *__restrict__ q,
               const int32_t *__restrict__ rows, const HistWork *__restrict__ work,
               const HistGroup *__restrict__ groups, int32_t n_groups,
               const int32_t *__restrict__ bin_ptr, int64_t total_bins,
               unsigned long long *__restrict__ hist, unsigned long long *__restrict__ n_updates)
{
    extern __shared__ unsigned long long lds[];
    const uint32_t L = xcd_remap(blockIdx.x, gridDim.x);
    const HistWork wk = work[L / n_groups];
    const HistGroup gr = groups[L % n_groups];
    const int32_t nb = gr.b1 - gr.b0;
    unsigned long long *sg = lds, *sh = lds + nb;
    for (int t = threadIdx.x; t < nb; t += kHistThreads) {
        sg[t] = 0ull;
        sh[t] = 0ull;
    }
    __syncthreads();
    unsigned int cnt = 0;
    for (int64_t i = wk.begin + threadIdx.x; i < wk.end; i += kHistThreads) {
        const int64_t r = kRows ? (int64_t)rows[i] : i;
        const longlong2 qq = q[r];
        const unsigned long long qg = (unsigned long long)qq.x, qh = (unsigned long long)qq.y;
        const uint32_t *p = page + r * row_words;
        if (!kSparse) {
            p += gr.w0;
            uint64_t buf = (uint64_t)(*p++) >> gr.skip;
            int32_t nbits = 32 - gr.skip;
            for (int32_t f = gr.f0; f < gr.f1; ++f) {
                if (nbits < w) {
                    buf |= (uint64_t)(*p++) << nbits;
                    nbits += 32;
                }
                const uint32_t sym = (uint32_t)buf & mask;
                buf >>= w;
                nbits -= w;
                if (sym != null_sym) {
                    const int32_t idx = bin_ptr[f] - gr.b0 + (int32_t)sym;
                    atomicAdd(&sg[idx], qg);
                    atomicAdd(&sh[idx], qh);
                    ++cnt;
                }
            }
        } else {
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
    }
    __syncthreads();
    unsigned long long *dst = hist + ((int64_t)wk.slot * total_bins + gr.b0) * 2;
    for (int t = threadIdx.x; t < nb; t += kHistThreads) {
        const unsigned long long g = sg[t], h = sh[t];
        if (g) atomicAdd(&dst[2 * t], g);
        if (h) atomicAdd(&dst[2 * t + 1], h);
    }
    if (n_updates) {
        for (int d = 32; d > 0; d >>= 1) cnt += __shfl_xor(cnt, d, 64);
        if ((threadIdx.x & 63) == 0 && cnt) atomicAdd(n_updates, (unsigned long long)cnt);
    }
}

__global__ void k_hist_zero(unsigned long long *__restrict__ hist, const int32_t *__restrict__ slots,
                            int64_t total_bins)
{
    const int64_t per = total_bins * 2;
    unsigned long long *h = hist + (int64_t)slots[blockIdx.y] * per;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < per;
         i += (int64_t)gridDim.x * blockDim.x)
        h[i] = 0ull;
}

__global__ void k_hist_sub(const longlong2 *__restrict__ parent, longlong2 *__restrict__ hist,
                           const gbt_sub *__restrict__ subs, int64_t total_bins)
{
    const gbt_sub s = subs[blockIdx.y];
    const longlong2 *p = parent + (int64_t)s.parent_slot * total_bins;
    const longlong2 *b = hist + (int64_t)s.built_slot * total_bins;
    longlong2 *t = hist + (int64_t)s.target_slot * total_bins;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total_bins;
         i += (int64_t)gridDim.x * blockDim.x) {
        longlong2 a = p[i], c = b[i];
        t[i] = make_longlong2(a.x - c.x, a.y - c.y);
    }
}

// Feature groups whose bins fit kLdsBins (a single wider feature gets a group
// of its own and the global-memory kernel).
static void make_groups(const gbt_matrix *mx, std::vector<HistGroup> *out, bool *fits)
{
    out->clear();
    *fits = true;
    int32_t f0 = 0;
    while (f0 < mx->m) {
        int32_t f1 = f0 + 1;
        while (f1 < mx->m && mx->bin_ptr_h[f1 + 1] - mx->bin_ptr_h[f0] <= kLdsBins) ++f1;
        HistGroup g;
        g.f0 = f0;
        g.f1 = f1;
        g.b0 = mx->bin_ptr_h[f0];
        g.b1 = mx->bin_ptr_h[f1];
        int64_t bit = (int64_t)f0 * mx->w;
        g.w0 = (int32_t)(bit >> 5);
        g.skip = (int32_t)(bit & 31);
        if (g.b1 - g.b0 > kLdsBins) *fits = false;
        out->push_back(g);
        f0 = f1;
    }
}

gbt_status build_hist_impl(gbt_ctx *c, const gbt_matrix *mx, const uint32_t *page, const int64_t *q,
                           const int32_t *rows, const gbt_seg *build, int32_t n_build,
                           const gbt_sub *sub, int32_t n_sub, const int64_t *parent_hist,
                           int64_t *hist, gbt_tree_stats *stats)
{
    const int64_t tb = mx->total_bins;
    if (tb == 0 || (n_build == 0 && n_sub == 0)) return GBT_OK;
    std::vector<HistGroup> groups;
    bool fits;
    make_groups(mx, &groups, &fits);
    if (!fits)
        return set_error(GBT_E_UNSUPPORTED, "a feature has more than %d bins", kLdsBins);
    const int32_t G = (int32_t)groups.size();

    int64_t total_rows = 0;
    for (int32_t k = 0; k < n_build; ++k) total_rows += std::max<int64_t>(0, build[k].end - build[k].begin);
    // chunk so the grid is a few waves of workgroups per CU
    const int64_t target_wg = 8 * kCUs;
    int64_t chunk = (total_rows * G + target_wg - 1) / target_wg;
    chunk = std::min<int64_t>(std::max<int64_t>(chunk, 2048), 1 << 20);
    std::vector<HistWork> work;
    std::vector<int32_t> slots;
    for (int32_t k = 0; k < n_build; ++k) {
        slots.push_back(build[k].node_slot);
        for (int64_t b = build[k].begin; b < build[k].end; b += chunk)
            work.push_back({b, std::min(build[k].end, b + chunk), build[k].node_slot, 0});
    }

    // upload the plan: groups | work | slots | subs
    size_t o_w = ((size_t)G * sizeof(HistGroup) + 255) / 256 * 256;
    size_t o_s = o_w + (work.size() * sizeof(HistWork) + 255) / 256 * 256;
    size_t o_u = o_s + (slots.size() * 4 + 255) / 256 * 256;
    size_t bytes = o_u + (size_t)n_sub * sizeof(gbt_sub) + 256;
    char *plan;
    GBT_TRY(scratch_t(c, kScrWork, bytes, &plan));
    std::vector<char> h(bytes);
    memcpy(h.data(), groups.data(), G * sizeof(HistGroup));
    if (!work.empty()) memcpy(h.data() + o_w, work.data(), work.size() * sizeof(HistWork));
    if (!slots.empty()) memcpy(h.data() + o_s, slots.data(), slots.size() * 4);
    if (n_sub) memcpy(h.data() + o_u, sub, (size_t)n_sub * sizeof(gbt_sub));
    GBT_HIP(hipMemcpyAsync(plan, h.data(), bytes, hipMemcpyHostToDevice, c->stream));
    const HistGroup *groups_d = (const HistGroup *)plan;
    const HistWork *work_d = (const HistWork *)(plan + o_w);
    const int32_t *slots_d = (const int32_t *)(plan + o_s);
    const gbt_sub *subs_d = (const gbt_sub *)(plan + o_u);

    unsigned long long *upd = nullptr;
    if (stats) GBT_TRY(scratch_t(c, kScrUpd, 1, &upd));

    if (n_build) {
        dim3 zg((unsigned)std::min<int64_t>((tb * 2 + 255) / 256, 1024), (unsigned)n_build);
        k_hist_zero<<<zg, 256, 0, c->stream>>>((unsigned long long *)hist, slots_d, tb);
        GBT_LAUNCHED();
    }
    if (!work.empty()) {
        if (stats) {
            unsigned long long zero = 0;
            GBT_HIP(hipMemcpyAsync(upd, &zero, 8, hipMemcpyHostToDevice, c->stream));
        }
        int32_t maxnb = 0;
        for (auto &g : groups) maxnb = std::max(maxnb, g.b1 - g.b0);
        size_t lds = (size_t)maxnb * 16;
        uint32_t null_sym = (mx->sparse || mx->has_missing) ? mx->null_sym : 0xffffffffu;
        uint32_t mask = mx->w >= 32 ? 0xffffffffu : ((1u << mx->w) - 1u);
        unsigned grid = (unsigned)(work.size() * (size_t)G);
        hipEvent_t e0 = nullptr, e1 = nullptr;
        if (c->timing && stats) {
            GBT_HIP(hipEventCreate(&e0));
            GBT_HIP(hipEventCreate(&e1));
            GBT_HIP(hipEventRecord(e0, c->stream));
        }
#define GBT_HIST_LAUNCH(SP, RW)                                                                    \
    k_hist_lds<SP, RW><<<grid, kHistThreads, lds, c->stream>>>(                                     \
        page, mx->row_words, mx->w, mask, null_sym, mx->stride, (const longlong2 *)q, rows, work_d, \
        groups_d, G, mx->bin_ptr_d, tb, (unsigned long long *)hist, upd)
        if (mx->sparse) {
            if (rows)
                GBT_HIST_LAUNCH(true, true);
            else
                GBT_HIST_LAUNCH(true, false);
        } else {
            if (rows)
                GBT_HIST_LAUNCH(false, true);
            else
                GBT_HIST_LAUNCH(false, false);
        }
#undef GBT_HIST_LAUNCH
        GBT_LAUNCHED();
        if (e0) {
            GBT_HIP(hipEventRecord(e1, c->stream));
            GBT_HIP(hipEventSynchronize(e1));
            float ms = 0.f;
            GBT_HIP(hipEventElapsedTime(&ms, e0, e1));
            stats->ms_hist += ms;
            (void)hipEventDestroy(e0);
            (void)hipEventDestroy(e1);
        }
        if (stats) {
            unsigned long long u = 0;
            GBT_HIP(hipMemcpyAsync(&u, upd, 8, hipMemcpyDeviceToHost, c->stream));
            GBT_HIP(hipStreamSynchronize(c->stream));
            int64_t wbytes = 4 * (((int64_t)mx->stride * mx->w + 31) / 32);
            stats->hist_launches += 1;
            stats->hist_rows += total_rows;
            stats->hist_updates += (int64_t)u;
            stats->hist_bytes += total_rows * (wbytes + 16 + (rows ? 4 : 0)) + (int64_t)n_build * tb * 16;
        }
    }
    if (n_sub) {
        GBT_CHECK(parent_hist, "subtraction needs the parent histograms");
        dim3 sg((unsigned)std::min<int64_t>((tb + 255) / 256, 1024), (unsigned)n_sub);
        k_hist_sub<<<sg, 256, 0, c->stream>>>((const longlong2 *)parent_hist, (longlong2 *)hist, subs_d, tb);
        GBT_LAUNCHED();
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
