// tree.hip -- one boosting iteration (Alg. 7 then Alg. 1 of the paper), the
// Eq. 6 leaves with the Eq. 1 margin update, Eq. 1 prediction, and the page
// streamer that feeds pinned-host ELLPACK pages to the device on a second
// stream, double buffered and overlapped with the kernels that consume them.
#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstring>
#include <functional>
#include <future>

#include "sample_impl.h"
#include "hist_impl.h"
#include "split_impl.h"
#include "plan_impl.h"

namespace gbt {

static unsigned blocks(int64_t n, int t = 256) { return (unsigned)((n + t - 1) / t); }

// ------------------------------------------------------------ page streamer
// Calls fn(words_d, row0, rows) for consecutive row chunks of every page.
// Device pages are passed in place; pinned-host pages are copied chunk by
// chunk on the side stream into two alternating device buffers, the copy of
// chunk c+1 overlapping the compute on chunk c.
using ChunkFn = std::function<gbt_status(const uint32_t *, int64_t, int64_t)>;

struct StreamEvents {
    hipEvent_t copied[2] = {nullptr, nullptr};
    hipEvent_t consumed[2] = {nullptr, nullptr};
    ~StreamEvents()
    {
        for (int i = 0; i < 2; ++i) {
            if (copied[i]) (void)hipEventDestroy(copied[i]);
            if (consumed[i]) (void)hipEventDestroy(consumed[i]);
        }
    }
};

gbt_status for_each_chunk(gbt_ctx *c, const gbt_matrix *mx, const ChunkFn &fn, double *h2d_bytes)
{
    struct Chunk {
        const GbtPage *pg;
        int64_t off, rows;
    };
    std::vector<Chunk> host_chunks;
    const int64_t chunk_rows = c->stream_chunk_rows;
    for (const auto &pg : mx->pages) {
        if (!pg.streamed()) {
            if (pg.rows) GBT_TRY(fn(pg.words, pg.row0, pg.rows));
            continue;
        }
        for (int64_t o = 0; o < pg.rows; o += chunk_rows)
            host_chunks.push_back({&pg, o, std::min(chunk_rows, pg.rows - o)});
    }
    if (host_chunks.empty()) return GBT_OK;
    const size_t row_bytes = (size_t)mx->row_words * 4;
    int64_t maxrows = 0;
    bool disk = false;
    for (auto &ch : host_chunks) {
        maxrows = std::max(maxrows, ch.rows);
        disk = disk || ch.pg->fd >= 0;
    }
    if (disk && c->disk_stage_bytes < (size_t)maxrows * row_bytes) {
        // pinned buffers the page files are read into (grow-only)
        GBT_HIP(hipStreamSynchronize(c->side));
        GBT_HIP(hipStreamSynchronize(c->stream));
        for (void *&p : c->disk_stage) {
            if (p) GBT_HIP(hipHostFree(p));
            p = nullptr;
        }
        c->disk_stage_bytes = 0;
        for (void *&p : c->disk_stage) GBT_HIP(hipHostMalloc(&p, (size_t)maxrows * row_bytes, hipHostMallocDefault));
        c->disk_stage_bytes = (size_t)maxrows * row_bytes;
    }
    uint32_t *buf[2];
    GBT_TRY(scratch(c, kScrStage0, (size_t)maxrows * row_bytes, (void **)&buf[0]));
    GBT_TRY(scratch(c, kScrStage1, (size_t)maxrows * row_bytes, (void **)&buf[1]));
    StreamEvents ev;
    for (int i = 0; i < 2; ++i) {
        GBT_HIP(hipEventCreateWithFlags(&ev.copied[i], hipEventDisableTiming));
        GBT_HIP(hipEventCreateWithFlags(&ev.consumed[i], hipEventDisableTiming));
    }
    // the buffers may still be read by earlier work on the compute stream
    GBT_HIP(hipEventRecord(ev.consumed[0], c->stream));
    GBT_HIP(hipEventRecord(ev.consumed[1], c->stream));
    GBT_HIP(hipEventRecord(ev.copied[0], c->side));
    GBT_HIP(hipEventRecord(ev.copied[1], c->side));
    // A disk chunk is first read into pinned buffer k & 1 by a worker
    // thread (once the copy of chunk k - 2 out of that buffer is done), so
    // that the file read overlaps the device's work on the chunk before it.
    std::future<gbt_status> reading;
    auto start_read = [&](size_t k) -> gbt_status {
        const Chunk &ch = host_chunks[k];
        int b = (int)(k & 1);
        GBT_HIP(hipEventSynchronize(ev.copied[b]));
        const int fd = ch.pg->fd;
        void *dst = c->disk_stage[b];
        const size_t bytes = (size_t)ch.rows * row_bytes;
        const int64_t off = ch.off * (int64_t)row_bytes;
        reading = std::async(std::launch::async, [=] {
            // in kReadParts pieces at once (page-aligned), this thread
            // reading the first
            constexpr size_t kReadParts = 8;
            if (bytes == 0) return GBT_OK;
            const size_t part = (bytes / kReadParts + 4095) & ~(size_t)4095;
            std::vector<std::future<gbt_status>> rest;
            for (size_t o = part; o < bytes; o += part)
                rest.push_back(std::async(std::launch::async, file_read, fd, (char *)dst + o,
                                          std::min(part, bytes - o), off + (int64_t)o));
            gbt_status s = file_read(fd, dst, std::min(part, bytes), off);
            for (auto &f : rest)
                if (f.get() != GBT_OK) s = GBT_E_IO;
            return s;
        });
        return GBT_OK;
    };
    auto issue = [&](size_t k) -> gbt_status {
        const Chunk &ch = host_chunks[k];
        int b = (int)(k & 1);
        const void *src = ch.pg->words + ch.off * mx->row_words;
        if (ch.pg->fd >= 0) {
            if (reading.get() != GBT_OK) return set_error(GBT_E_IO, "reading a page file failed");
            src = c->disk_stage[b];
        }
        GBT_HIP(hipStreamWaitEvent(c->side, ev.consumed[b], 0));
        GBT_HIP(hipMemcpyAsync(buf[b], src, (size_t)ch.rows * row_bytes, hipMemcpyHostToDevice, c->side));
        GBT_HIP(hipEventRecord(ev.copied[b], c->side));
        if (h2d_bytes) *h2d_bytes += (double)ch.rows * row_bytes;
        return GBT_OK;
    };
    auto on_disk = [&](size_t k) { return host_chunks[k].pg->fd >= 0; };
    if (on_disk(0)) GBT_TRY(start_read(0));
    GBT_TRY(issue(0));
    for (size_t k = 0; k < host_chunks.size(); ++k) {
        const bool next = k + 1 < host_chunks.size();
        // pinned chunks: the next copy goes out before this chunk's work;
        // disk chunks: the next read runs during it, its copy after it
        if (next) GBT_TRY(on_disk(k + 1) ? start_read(k + 1) : issue(k + 1));
        int b = (int)(k & 1);
        GBT_HIP(hipStreamWaitEvent(c->stream, ev.copied[b], 0));
        const Chunk &ch = host_chunks[k];
        GBT_TRY(fn(buf[b], ch.pg->row0 + ch.off, ch.rows));
        GBT_HIP(hipEventRecord(ev.consumed[b], c->stream));
        if (next && on_disk(k + 1)) GBT_TRY(issue(k + 1));
    }
    // keep the events alive until the side stream is done with them
    GBT_HIP(hipStreamSynchronize(c->side));
    return GBT_OK;
}

// Holds the staging buffers for_each_chunk uses for mx's pinned pages, so
// that later workspaces sized by the remaining budget leave room for them.
static gbt_status reserve_stage(gbt_ctx *c, const gbt_matrix *mx)
{
    int64_t maxrows = 0;
    for (const auto &pg : mx->pages)
        if (pg.streamed()) maxrows = std::max(maxrows, std::min(pg.rows, c->stream_chunk_rows));
    if (maxrows == 0) return GBT_OK;
    void *p;
    GBT_TRY(scratch(c, kScrStage0, (size_t)maxrows * mx->row_words * 4, &p));
    GBT_TRY(scratch(c, kScrStage1, (size_t)maxrows * mx->row_words * 4, &p));
    return GBT_OK;
}

static bool all_device_single(const gbt_matrix *mx)
{
    return mx->pages.size() == 1 && !mx->pages[0].streamed();
}

static bool any_host_pages(const gbt_matrix *mx)
{
    for (auto &pg : mx->pages)
        if (pg.streamed()) return true;
    return false;
}

// ------------------------------------------------------------ sampling driver
struct Buffers {
    gbt_ctx *c;
    bool owned;
    std::vector<std::pair<void *, size_t>> held;
    gbt_status get(int slot, size_t bytes, void **p)
    {
        if (!owned) return scratch(c, slot, bytes, p);
        GBT_TRY(dev_alloc(c, bytes, p));
        held.push_back({*p, bytes});
        return GBT_OK;
    }
    void release()
    {
        for (auto &h : held) dev_free(c, h.first, h.second);
        held.clear();
    }
};

struct SampleOut {
    const uint32_t *page = nullptr;  // R rows
    int32_t *sel = nullptr;          // R global ids (NULL: identity)
    double *gw = nullptr;
    int64_t *q = nullptr;
    int64_t R = 0, K = 0, T = 0;
    int32_t e_key = 0, e_g = 0, e_h = 0;
    bool alias = false;
    long long root_g = 0, root_h = 0;
    SampleState *st = nullptr;
};

// The lambda of the sampling keys: 0 for GOSS (keys are |g|).
static double sample_lambda(const gbt_sample_params &sp)
{
    return sp.sampler == GBT_SAMPLE_GOSS && sp.f < 1.0 ? 0.0 : sp.mvs_lambda;
}

// Alg. 7: g' <- Sample(g); AllocateOnGPU(sampled_page); Compact each page.
// st_ready: the caller has initialized st and folded the maximum of r into
// it while computing the gradients.  read_state: copy the threshold,
// exponents and root sums to the host (o->T ... o->root_h); otherwise they
// stay in o->st on the device.
gbt_status sample_run(gbt_ctx *c, const gbt_matrix *mx, const float *gpair, const float *margin,
                      const float *label, const gbt_sample_params &sp, Buffers &bufs, SampleOut *o,
                      double *h2d_bytes, SampleState *st_ready = nullptr, bool read_state = true,
                      bool keys_spec = false)
{
    const int64_t n = mx->n_rows;
    GBT_CHECK(sp.f > 0.0 && sp.f <= 1.0, "sampling fraction %g outside (0, 1]", sp.f);
    GBT_CHECK(sp.sampler >= GBT_SAMPLE_MVS && sp.sampler <= GBT_SAMPLE_GOSS, "unknown sampler %d", sp.sampler);
    GBT_CHECK(sp.sampler != GBT_SAMPLE_GOSS || sp.f >= 1.0 ||
                  (sp.goss_a >= 0.0 && sp.goss_a < 1.0 && sp.f - sp.goss_a > 0.0),
              "GOSS needs 0 <= a < 1 and a < f (a = %g, f = %g)", sp.goss_a, sp.f);
    // GOSS ranks rows by |g|: its keys are the MVS keys with lambda = 0
    const double lam = sample_lambda(sp);
    SampleRule rule{GBT_SAMPLE_MVS, 0, 0, 1.0};
    GBT_CHECK(gpair || (margin && label), "sampling needs gradient pairs or margins and labels");
    SampleState *st = st_ready;
    if (!st) {
        GBT_TRY(bufs.get(kScrState, sizeof(SampleState), (void **)&st));
        GBT_TRY(state_init(c, st));
    }
    o->st = st;
    SampleSrc src{(const float2 *)gpair, margin, label, sp.loss, 0};
    const int kind = gpair ? kSrcGpair : kSrcMargin;
    bool fx_max_done = false;

    if (sp.f >= 1.0 && all_device_single(mx) && gpair) {
        // no sampling: the data page trains as it is
        o->alias = true;
        o->page = mx->pages[0].words;
        o->R = n;
        GBT_TRY(bufs.get(kScrGw, (size_t)std::max<int64_t>(n, 1) * 16, (void **)&o->gw));
        GBT_TRY(gw_all(c, gpair, n, o->gw));
    } else {
        uint8_t *keep;
        int32_t *tile_off;
        const int64_t ntiles = (n + kCompactTile - 1) / kCompactTile;
        GBT_TRY(bufs.get(kScrFlags, (size_t)std::max<int64_t>(n, 16) + 16, (void **)&keep));
        GBT_TRY(bufs.get(kScrPos, (size_t)(ntiles + 1) * 4, (void **)&tile_off));
        // a draw passes with probability p < 1 when U < floor(p 2^64)
        auto draw_limit = [](double p) -> uint64_t { return (uint64_t)std::ldexp(p, 64); };
        if (sp.f < 1.0 && sp.sampler == GBT_SAMPLE_SGB) {
            rule = SampleRule{GBT_SAMPLE_SGB, 0, draw_limit(sp.f), 1.0};
        } else if (sp.f < 1.0 && sp.sampler == GBT_SAMPLE_GOSS) {
            const double a = sp.goss_a, b = sp.f - sp.goss_a, p = b / (1.0 - a);
            o->K = std::min<int64_t>(n, std::max<int64_t>(0, (int64_t)std::nearbyint(a * (double)n)));
            GBT_TRY(mvs_threshold(c, src, kind, nullptr, n, lam, o->K, st, true, st_ready != nullptr, true));
            rule = SampleRule{GBT_SAMPLE_GOSS, p >= 1.0 ? 1 : 0, p >= 1.0 ? 0 : draw_limit(p), (1.0 - a) / b};
        }
        // MVS: the selection is queued right behind the threshold's first
        // kernel, before the host learns whether the closed form held (it
        // almost always does); otherwise the threshold is completed and the
        // selection queued again
        const bool mvs = sp.f < 1.0 && sp.sampler == GBT_SAMPLE_MVS;
        // the threshold's first step is made by the selection's blocks
        ThreshFuse fuse;
        if (mvs) {
            o->K = std::max<int64_t>(1, (int64_t)std::nearbyint(sp.f * (double)n));
            GBT_TRY(mvs_threshold(c, src, kind, nullptr, n, lam, o->K, st, true, st_ready != nullptr, false,
                                  keys_spec && st_ready != nullptr, true, n > 0 ? &fuse : nullptr));
        }
        // the sample size sizes the buffers below: one round trip (its word
        // sits apart from the threshold's flag in the pinned buffer)
        void *hio, *hio_d;
        GBT_TRY(host_io(c, 64, &hio, &hio_d));
        volatile int32_t *r_host = (volatile int32_t *)hio + 4;
        // scan: the tile offsets by a scan of their own (else the early
        // compaction sums the counts itself)
        auto select = [&](bool wait, bool scan) -> gbt_status {
            // with f = 1 the state keeps T = 0: every row is kept with weight 1
            *r_host = -1;
            GBT_TRY(mvs_select(c, src, kind, nullptr, n, lam, st, sp.seed, sp.iteration, 0, keep, tile_off, rule,
                               fuse));
            fuse = ThreshFuse{};  // a selection queued again reads the completed threshold
            if (scan) GBT_TRY(keep_tile_offsets(c, n, tile_off, (int32_t *)hio_d + 4));
            if (wait) GBT_HIP(hipStreamSynchronize(c->stream));
            return GBT_OK;
        };
        const size_t rb = (size_t)mx->row_words * 4;
        // A page on the device with the context's own workspaces: the
        // compaction is queued behind the selection before the host reads
        // the sample size, into buffers sized for about f n rows (held from
        // the trees before), so the host's round trip overlaps it.  It is
        // redone when the threshold had to be completed or the sample is
        // larger than the buffers.
        const bool early = all_device_single(mx) && !bufs.owned && n > 0 && !(mvs && c->mvs_descent_last);
        int64_t cap = 0;
        uint32_t *spage = nullptr;
        if (early) {
            const int64_t guess = std::min<int64_t>(n, (int64_t)std::ceil(sp.f * (double)n)) + 1;
            GBT_TRY(bufs.get(kScrSampled, (size_t)guess * rb, (void **)&spage));
            GBT_TRY(bufs.get(kScrSel, (size_t)guess * 4, (void **)&o->sel));
            GBT_TRY(bufs.get(kScrGw, (size_t)guess * 16, (void **)&o->gw));
            cap = (int64_t)std::min({scratch_bytes(c, kScrSampled) / rb, scratch_bytes(c, kScrSel) / 4,
                                     scratch_bytes(c, kScrGw) / 16});
            GBT_TRY(select(false, false));
            GBT_TRY(mvs_compact_tiles(c, src, kind, n, lam, st, keep, tile_off, 0, n, mx->pages[0].words,
                                      mx->row_words, spage, o->sel, o->gw, rule, cap, (int32_t *)hio_d + 4));
            GBT_TRY(wait_flag(c, r_host));
        } else {
            GBT_TRY(select(true, true));
        }
        bool redo = false;
        if (mvs) {
            GBT_TRY(mvs_threshold_resume(c, src, kind, nullptr, n, lam, o->K, st, &redo));
            // the threshold's flag: 1 closed form, 0 the descent ran
            c->mvs_descent_last = redo && *(volatile int32_t *)hio == 0;
            if (redo) GBT_TRY(select(true, true));
        }
        o->R = *r_host;
        GBT_CHECK(o->R >= 0 && o->R <= n, "sample size %lld of %lld rows", (long long)o->R, (long long)n);
        const bool compacted = early && !redo && o->R <= cap;
        // the early compaction's maxima of the reweighted pairs are void;
        // its tile counts (when no selection was queued again) become offsets
        if (early && !compacted) GBT_TRY(fx_max_reset(c, st));
        if (early && !compacted && !redo) GBT_TRY(keep_tile_offsets(c, n, tile_off, nullptr));
        GBT_TRY(bufs.get(kScrSampled, (size_t)std::max<int64_t>(o->R, 1) * rb, (void **)&spage));
        GBT_TRY(bufs.get(kScrSel, (size_t)std::max<int64_t>(o->R, 1) * 4, (void **)&o->sel));
        GBT_TRY(bufs.get(kScrGw, (size_t)std::max<int64_t>(o->R, 1) * 16, (void **)&o->gw));
        o->page = spage;
        // (disk pages have no device mapping: they always stream)
        const bool host = any_host_pages(mx) && mx->page_home == GBT_HOME_PINNED_HOST;
        const bool gather = host && (c->compaction == GBT_COMPACT_GATHER ||
                                     (c->compaction == GBT_COMPACT_AUTO && 2 * (int64_t)o->R <= n));
        if (compacted) {
        } else if (gather) {
            // the kernel reads the kept rows of each pinned page through its
            // device mapping: only those rows cross the host link
            for (const auto &pg : mx->pages) {
                if (!pg.rows) continue;
                const uint32_t *w = pg.words;
                if (pg.host) {
                    void *dp = nullptr;
                    GBT_HIP(hipHostGetDevicePointer(&dp, (void *)pg.words, 0));
                    GBT_CHECK(dp != nullptr, "no device mapping of a pinned page");
                    w = (const uint32_t *)dp;
                }
                GBT_TRY(mvs_compact_tiles(c, src, kind, n, lam, st, keep, tile_off, pg.row0, pg.row0 + pg.rows, w,
                                          mx->row_words, spage, o->sel, o->gw, rule));
            }
            // every page of a matrix has the same home
            if (h2d_bytes) *h2d_bytes += (double)o->R * (double)rb;
            // the margin update still streams every page
            GBT_TRY(reserve_stage(c, mx));
        } else {
            GBT_TRY(for_each_chunk(
                c, mx,
                [&](const uint32_t *words, int64_t row0, int64_t rows) -> gbt_status {
                    return mvs_compact_tiles(c, src, kind, n, lam, st, keep, tile_off, row0, row0 + rows,
                                             words, mx->row_words, spage, o->sel, o->gw, rule);
                },
                h2d_bytes));
        }
        fx_max_done = true;
    }
    GBT_TRY(bufs.get(kScrQ, (size_t)std::max<int64_t>(o->R, 1) * 16, (void **)&o->q));
    GBT_TRY(fixed_point(c, o->gw, o->R, st, o->q, fx_max_done));
    if (!read_state) return GBT_OK;
    SampleState hst;
    GBT_HIP(hipMemcpyAsync(&hst, st, sizeof(SampleState), hipMemcpyDeviceToHost, c->stream));
    GBT_HIP(hipStreamSynchronize(c->stream));
    if (hst.bad) return set_error(GBT_E_INVALID, "sampling failed (state flags %u)", hst.bad);
    o->T = hst.T;
    o->e_key = hst.e_key;
    o->e_g = hst.e_g;
    o->e_h = hst.e_h;
    o->root_g = (long long)fold_sum(hst.root_g);
    o->root_h = (long long)fold_sum(hst.root_h);
    return GBT_OK;
}

// ------------------------------------------------------------ tree kernels
// The node table, the root (its sums from the sampling state), the root
// level list and counts, the root histogram's work (R rows in chunks of
// `chunk`, n_root items, summed into slot 0), the identity slot order, and
// zeroed counters (histogram updates, level statistics).
__global__ void k_tree_init(DevNode *__restrict__ nodes, int32_t n_nodes, const SampleState *__restrict__ st,
                            int64_t R, EvalNode *__restrict__ level, int32_t *__restrict__ cnt,
                            HistWork *__restrict__ work, HistReduce *__restrict__ red, int64_t chunk,
                            int32_t n_root, int32_t *__restrict__ rows, int32_t *__restrict__ slot_node,
                            int64_t n_slots, unsigned long long *__restrict__ upd,
                            unsigned long long *__restrict__ stat)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n_slots) {  // the root's slots (the root level's partition does not read them)
        rows[i] = (int32_t)i;
        slot_node[i] = 0;
    }
    if (upd && i < kUpdCounters) upd[i * kUpdStride] = 0ull;
    if (i < 2) stat[i] = 0ull;
    if (i < n_nodes) {
        DevNode d;
        memset(&d, 0, sizeof(d));
        d.left_child = 2 * (int32_t)i + 1;
        d.right_child = 2 * (int32_t)i + 2;
        if (i == 0) {
            const long long rg = (long long)fold_sum(st->root_g), rh = (long long)fold_sum(st->root_h);
            d.present = 1;
            d.sum_g = rg;
            d.sum_h = rh;
            d.begin = 0;
            d.end = R;
            level[0] = {rg, rh, 0, 0};
            cnt[0] = 1;
            cnt[1] = cnt[2] = cnt[3] = 0;
            red[0] = {0, 0, n_root, -1, -1, 0};
        }
        nodes[i] = d;
    }
    if (i < n_root) {
        const int64_t b = i * chunk;
        work[i] = {b, b + chunk < R ? b + chunk : R, (int32_t)i, 0};
    }
}

// Leaf values and the compact tree, when the last level's plan did not make
// them (no level, or no rows).
__global__ void k_leaves(const DevNode *__restrict__ nodes, int32_t n_nodes, const int32_t *__restrict__ e_dev,
                         double lambda, double eta, float *__restrict__ leaf, uint2 *__restrict__ compact)
{
    int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n_nodes) return;
    leaf_entry(nodes, i, e_dev[0], e_dev[1], lambda, eta, leaf, compact);
}

// What the host reads after a tree, written by the device into pinned memory.
struct TreeResult {
    unsigned long long updates;     // histogram updates (the counters folded)
    unsigned long long rows_built;  // rows streamed below the root
    unsigned long long built;       // histograms built below the root
    long long T;
    int32_t e_key, e_g, e_h;
    uint32_t bad;
    gbt_node nodes[1];  // n_nodes entries
};

// The tree in its public form (threshold = the split's cut value) and the
// call's counters, written into the host's pinned result.
struct FinalizeArgs {
    const DevNode *nodes;
    int32_t n_nodes;
    int32_t pad0;
    const float *leaf;
    const int32_t *cut_ptr;
    const float *cut_values;
    const SampleState *st;
    const unsigned long long *upd;
    const unsigned long long *stat;
    TreeResult *out;
    SampleState *reset;  // when not NULL: st, reset for the next tree once read
};

__device__ inline void finalize_entry(const FinalizeArgs &a, int32_t i)
{
    if (i == 0) {
        unsigned long long u = 0;
        if (a.upd)
            for (int k = 0; k < kUpdCounters; ++k) u += a.upd[k * kUpdStride];
        a.out->updates = u;
        a.out->rows_built = a.stat[0];
        a.out->built = a.stat[1];
        a.out->T = a.st->T;
        a.out->e_key = a.st->e_key;
        a.out->e_g = a.st->e_g;
        a.out->e_h = a.st->e_h;
        a.out->bad = a.st->bad;
    }
    if (i >= a.n_nodes) return;
    const DevNode d = a.nodes[i];
    gbt_node o;
    memset(&o, 0, sizeof(o));
    if (d.present) {
        o.flags = GBT_NODE_PRESENT;
        o.sum_g = d.sum_g;
        o.sum_h = d.sum_h;
        o.n_rows = (int32_t)(d.end - d.begin);
        if (d.split) {
            o.feature = d.feature;
            o.split_bin = d.split_bin;
            o.threshold = a.cut_values[a.cut_ptr[d.feature] + d.split_bin - 1];
            o.gain = d.gain;
            if (d.default_left) o.flags |= GBT_NODE_DEFAULT_LEFT;
        } else {
            o.feature = -1;
            o.split_bin = -1;
            o.flags |= GBT_NODE_LEAF;
            o.leaf_value = a.leaf[i];
        }
    }
    a.out->nodes[i] = o;  // absent nodes stay all zero
}

// The block of entry 0 (the only reader of the sampling state) resets the
// state afterwards when asked.
__device__ inline void finalize_block(const FinalizeArgs &a, uint32_t b)
{
    finalize_entry(a, (int32_t)(b * blockDim.x + threadIdx.x));
    if (a.reset && b == 0) {
        __syncthreads();  // entry 0 has read the state
        state_reset_block(a.reset);
    }
}

__global__ void k_finalize(FinalizeArgs a) { finalize_block(a, blockIdx.x); }

// Margin update from the final node of each training slot (no sampling:
// the slots hold every row once).
__global__ void k_margin_slots(float *__restrict__ margin, const int32_t *__restrict__ rows,
                               const int32_t *__restrict__ slot_node, const float *__restrict__ leaf, int64_t n)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const int32_t r = rows[i];
    margin[r] = margin[r] + leaf[slot_node[i]];
}

// Row staging for the tree walks: the block's 256 consecutive rows are read
// with coalesced 16-byte loads into LDS (row stride padded to an odd word
// count against bank conflicts); each lane then walks its row from LDS.
constexpr int kWalkThreads = 256;
constexpr int kWalkMaxWords = 60;  // rows up to this many words are staged

template <bool kStage>
__device__ inline const uint32_t *stage_row(const uint32_t *__restrict__ words, int64_t rows,
                                            int32_t row_words, uint32_t *lds)
{
    const int64_t r0 = (int64_t)blockIdx.x * kWalkThreads;
    if (!kStage) return words + (r0 + threadIdx.x) * row_words;
    const int32_t ps = row_words + 1;
    const int32_t q4 = row_words / 4;
    const int32_t nr = (int32_t)min((int64_t)kWalkThreads, rows - r0);
    const uint4 *src = (const uint4 *)(words + r0 * row_words);
    for (int32_t t = threadIdx.x; t < nr * q4; t += kWalkThreads) {
        uint4 v = src[t];
        uint32_t *d = lds + (t / q4) * ps + (t % q4) * 4;
        d[0] = v.x;
        d[1] = v.y;
        d[2] = v.z;
        d[3] = v.w;
    }
    __syncthreads();
    return lds + threadIdx.x * ps;
}

// Margin update by walking each row's symbols down the tree.
template <bool kStage>
__global__ void __launch_bounds__(kWalkThreads)
    k_margin_walk(const uint32_t *__restrict__ words, int64_t rows, Geo geo,
                  const DevNode *__restrict__ nodes, const float *__restrict__ leaf,
                  float *__restrict__ margin)
{
    extern __shared__ __align__(16) uint32_t walk_lds[];
    const uint32_t *row = stage_row<kStage>(words, rows, geo.row_words, walk_lds);
    int64_t i = (int64_t)blockIdx.x * kWalkThreads + threadIdx.x;
    if (i >= rows) return;
    int32_t id = 0;
    while (nodes[id].split) {
        const DevNode &d = nodes[id];
        int32_t b = row_feature_bin(row, geo, d.feature);
        bool left = b < 0 ? d.default_left != 0 : b < d.split_bin;
        id = left ? d.left_child : d.right_child;
    }
    margin[i] = margin[i] + leaf[id];
}

// Margin update of every row by walking the tree held in LDS.  The grid is
// a few blocks per CU; each block loads the compact tree once, then loops
// over tiles of 256 rows staged through LDS with coalesced loads.
constexpr int kWalkTileRows = 256;
constexpr int kWalkLdsNodes = 4095;  // trees up to depth 11 are held in LDS

__global__ void __launch_bounds__(kWalkTileRows)
    k_margin_walk_lds(const uint32_t *__restrict__ words, int64_t rows, Geo geo,
                      const uint2 *__restrict__ compact, const float *__restrict__ leaf, int32_t nn,
                      float *__restrict__ margin)
{
    extern __shared__ __align__(16) uint32_t walk_lds[];
    uint2 *tn = (uint2 *)walk_lds;
    float *tl = (float *)(tn + nn);
    uint32_t *rb = (uint32_t *)(tl + nn);
    for (int32_t t = threadIdx.x; t < nn; t += kWalkTileRows) {
        tn[t] = compact[t];
        tl[t] = leaf[t];
    }
    const int32_t ps = geo.row_words + 1, q4 = geo.row_words / 4;
    const int64_t n_tiles = (rows + kWalkTileRows - 1) / kWalkTileRows;
    for (int64_t tile = blockIdx.x; tile < n_tiles; tile += gridDim.x) {
        const int64_t r0 = tile * kWalkTileRows;
        const int32_t nr = (int32_t)min((int64_t)kWalkTileRows, rows - r0);
        const uint4 *src = (const uint4 *)(words + r0 * geo.row_words);
        __syncthreads();  // the previous tile's rows are consumed
        for (int32_t t = threadIdx.x; t < nr * q4; t += kWalkTileRows) {
            uint4 v = src[t];
            uint32_t *d = rb + (t / q4) * ps + (t % q4) * 4;
            d[0] = v.x;
            d[1] = v.y;
            d[2] = v.z;
            d[3] = v.w;
        }
        __syncthreads();
        if ((int32_t)threadIdx.x < nr) {
            const uint32_t *row = rb + threadIdx.x * ps;
            int32_t id = 0;
            uint2 nd = tn[0];
            while (nd.y & 1u) {
                int32_t b = row_feature_bin(row, geo, (int32_t)nd.x);
                bool left = b < 0 ? ((nd.y >> 1) & 1u) != 0 : b < (int32_t)(nd.y >> 2);
                id = 2 * id + (left ? 1 : 2);
                nd = tn[id];
            }
            const int64_t i = r0 + threadIdx.x;
            margin[i] = margin[i] + tl[id];
        }
    }
}

// The same walk with the next tile's rows and margins prefetched into
// registers (kQ 16-byte pieces per row) while the current tile is walked.
// Dense rows: the tree in LDS holds each split's bit offset (feature * w),
// and a symbol is one funnel shift of two words of the staged row (the row
// pitch leaves a word after the last one).
template <int kQ>
__global__ void __launch_bounds__(kWalkTileRows)
    k_margin_walk_pf(const uint32_t *__restrict__ words, int64_t rows, Geo geo,
                     const uint2 *__restrict__ compact, const float *__restrict__ leaf, int32_t nn,
                     float *__restrict__ margin, int32_t fin_blocks, FinalizeArgs fa)
{
    // the last fin_blocks blocks write the tree's host result instead
    const uint32_t walk_blocks = gridDim.x - (uint32_t)fin_blocks;
    if (blockIdx.x >= walk_blocks) {
        finalize_block(fa, blockIdx.x - walk_blocks);
        return;
    }
    extern __shared__ __align__(16) uint32_t walk_lds[];
    uint2 *tn = (uint2 *)walk_lds;
    float *tl = (float *)(tn + nn);
    uint32_t *rb = (uint32_t *)(tl + nn);
    const bool dense = !geo.sparse;
    constexpr int32_t ps = 4 * kQ + 1;  // odd row pitch in LDS
    const int64_t n_tiles = (rows + kWalkTileRows - 1) / kWalkTileRows;
    uint4 nxt[kQ];
    float mnext = 0.0f;
    auto load = [&](int64_t tile) {
        const int64_t r0 = tile * kWalkTileRows;
        const int32_t nr = (int32_t)min((int64_t)kWalkTileRows, rows - r0);
        const uint4 *src = (const uint4 *)(words + r0 * geo.row_words);
#pragma unroll
        for (int j = 0; j < kQ; ++j) {
            const int32_t e = threadIdx.x + j * kWalkTileRows;
            nxt[j] = e < nr * kQ ? src[e] : make_uint4(0u, 0u, 0u, 0u);
        }
        mnext = (int32_t)threadIdx.x < nr ? margin[r0 + threadIdx.x] : 0.0f;
    };
    // the first tile's rows are requested before the tree, so that their
    // trip to memory overlaps the tree's (cached) loads
    int64_t tile = blockIdx.x;
    if (tile < n_tiles) load(tile);
    for (int32_t t = threadIdx.x; t < nn; t += kWalkTileRows) {
        uint2 c = compact[t];
        if (dense && (c.y & 1u)) c.x *= (uint32_t)geo.w;
        tn[t] = c;
        tl[t] = leaf[t];
    }
    for (; tile < n_tiles; tile += walk_blocks) {
        const int64_t r0 = tile * kWalkTileRows;
        const int32_t nr = (int32_t)min((int64_t)kWalkTileRows, rows - r0);
        __syncthreads();  // the previous tile's rows are consumed (and the tree is loaded)
#pragma unroll
        for (int j = 0; j < kQ; ++j) {
            const int32_t e = threadIdx.x + j * kWalkTileRows;
            uint32_t *d = rb + (e / kQ) * ps + (e % kQ) * 4;
            d[0] = nxt[j].x;
            d[1] = nxt[j].y;
            d[2] = nxt[j].z;
            d[3] = nxt[j].w;
        }
        const float m = mnext;
        __syncthreads();
        if (tile + walk_blocks < n_tiles) load(tile + walk_blocks);
        if ((int32_t)threadIdx.x < nr) {
            const uint32_t *row = rb + threadIdx.x * ps;
            int32_t id = 0;
            uint2 nd = tn[0];
            if (dense) {
                while (nd.y & 1u) {
                    const uint32_t k = nd.x >> 5;
                    const uint32_t sym = __builtin_amdgcn_alignbit(row[k + 1], row[k], nd.x & 31u) & geo.mask;
                    const bool left = sym == geo.null_sym ? ((nd.y >> 1) & 1u) != 0 : sym < (nd.y >> 2);
                    id = 2 * id + (left ? 1 : 2);
                    nd = tn[id];
                }
            } else {
                while (nd.y & 1u) {
                    const int32_t b = row_feature_bin(row, geo, (int32_t)nd.x);
                    const bool left = b < 0 ? ((nd.y >> 1) & 1u) != 0 : b < (int32_t)(nd.y >> 2);
                    id = 2 * id + (left ? 1 : 2);
                    nd = tn[id];
                }
            }
            margin[r0 + threadIdx.x] = m + tl[id];
        }
    }
}

// grid walk blocks, then fin_blocks blocks of the tree's host result (fa)
static void launch_walk_pf(gbt_ctx *c, int q4, unsigned grid, size_t lds_bytes, const uint32_t *words,
                           int64_t rows, const Geo &geo, const uint2 *compact, const float *leaf, int32_t nn,
                           float *margin, int32_t fin_blocks, const FinalizeArgs &fa)
{
#define GBT_WALK_PF(Q)                                                                                         \
    case Q:                                                                                                    \
        k_margin_walk_pf<Q><<<grid + (unsigned)fin_blocks, kWalkTileRows, lds_bytes, c->stream>>>(              \
            words, rows, geo, compact, leaf, nn, margin, fin_blocks, fa);                                      \
        break;
    switch (q4) {
        GBT_WALK_PF(1)
        GBT_WALK_PF(2)
        GBT_WALK_PF(3)
        GBT_WALK_PF(4)
        GBT_WALK_PF(5)
        GBT_WALK_PF(6)
        GBT_WALK_PF(7)
        GBT_WALK_PF(8)
    }
#undef GBT_WALK_PF
}

// ------------------------------------------------------------ prediction
__device__ inline int32_t walk_binned(const gbt_node *__restrict__ t, int64_t nn, const uint32_t *row,
                                      const Geo &geo)
{
    int32_t id = 0;
    while (!(t[id].flags & GBT_NODE_LEAF) && 2 * (int64_t)id + 2 < nn) {
        int32_t b = row_feature_bin(row, geo, t[id].feature);
        bool left = b < 0 ? (t[id].flags & GBT_NODE_DEFAULT_LEFT) != 0 : b < t[id].split_bin;
        id = left ? 2 * id + 1 : 2 * id + 2;
    }
    return id;
}

template <bool kStage>
__global__ void __launch_bounds__(kWalkThreads)
    k_predict_binned(const uint32_t *__restrict__ words, int64_t rows, Geo geo,
                     const gbt_node *__restrict__ trees, const int64_t *__restrict__ offs,
                     int32_t n_trees, float base, float *__restrict__ out)
{
    extern __shared__ __align__(16) uint32_t walk_lds[];
    const uint32_t *row = stage_row<kStage>(words, rows, geo.row_words, walk_lds);
    int64_t i = (int64_t)blockIdx.x * kWalkThreads + threadIdx.x;
    if (i >= rows) return;
    float acc = base;
    for (int32_t t = 0; t < n_trees; ++t) {
        const gbt_node *tr = trees + offs[t];
        acc = acc + tr[walk_binned(tr, offs[t + 1] - offs[t], row, geo)].leaf_value;
    }
    out[i] = acc;
}

__global__ void k_predict_raw_dense(const float *__restrict__ X, int64_t n, int64_t ld,
                                    const gbt_node *__restrict__ trees, const int64_t *__restrict__ offs,
                                    int32_t n_trees, float base, float *__restrict__ out)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const float *x = X + i * ld;
    float acc = base;
    for (int32_t t = 0; t < n_trees; ++t) {
        const gbt_node *tr = trees + offs[t];
        const int64_t nn = offs[t + 1] - offs[t];
        int32_t id = 0;
        while (!(tr[id].flags & GBT_NODE_LEAF) && 2 * (int64_t)id + 2 < nn) {
            float v = x[tr[id].feature];
            bool left = v != v ? (tr[id].flags & GBT_NODE_DEFAULT_LEFT) != 0 : v <= tr[id].threshold;
            id = left ? 2 * id + 1 : 2 * id + 2;
        }
        acc = acc + tr[id].leaf_value;
    }
    out[i] = acc;
}

__global__ void k_predict_raw_csr(const int64_t *__restrict__ indptr, const int32_t *__restrict__ idx,
                                  const float *__restrict__ val, int64_t n,
                                  const gbt_node *__restrict__ trees, const int64_t *__restrict__ offs,
                                  int32_t n_trees, float base, float *__restrict__ out)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    int64_t base_e = indptr[0];
    int64_t e0 = indptr[i] - base_e, e1 = indptr[i + 1] - base_e;
    float acc = base;
    for (int32_t t = 0; t < n_trees; ++t) {
        const gbt_node *tr = trees + offs[t];
        const int64_t nn = offs[t + 1] - offs[t];
        int32_t id = 0;
        while (!(tr[id].flags & GBT_NODE_LEAF) && 2 * (int64_t)id + 2 < nn) {
            int32_t j = tr[id].feature;
            float v = __builtin_nanf("");
            int64_t lo = e0, hi = e1;  // binary search: indices ascend
            while (lo < hi) {
                int64_t mid = (lo + hi) >> 1;
                if (idx[mid] < j)
                    lo = mid + 1;
                else
                    hi = mid;
            }
            if (lo < e1 && idx[lo] == j) v = val[lo];
            bool left = v != v ? (tr[id].flags & GBT_NODE_DEFAULT_LEFT) != 0 : v <= tr[id].threshold;
            id = left ? 2 * id + 1 : 2 * id + 2;
        }
        acc = acc + tr[id].leaf_value;
    }
    out[i] = acc;
}

__global__ void k_leaf_values(gbt_node *__restrict__ t, int32_t n, int32_t eg, int32_t eh, double lambda,
                              double eta)
{
    int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    if ((t[i].flags & GBT_NODE_PRESENT) && (t[i].flags & GBT_NODE_LEAF))
        t[i].leaf_value = leaf_of(t[i].sum_g, t[i].sum_h, eg, eh, lambda, eta);
}

// Rows whose leaf is known (bit r of done, global row row0 + i): skipped.
template <bool kStage>
__global__ void __launch_bounds__(kWalkThreads)
    k_margin_add_tree(const uint32_t *__restrict__ words, int64_t rows, Geo geo,
                      const gbt_node *__restrict__ t, int64_t nn, float *__restrict__ margin,
                      const uint32_t *__restrict__ done, int64_t row0)
{
    extern __shared__ __align__(16) uint32_t walk_lds[];
    const uint32_t *row = stage_row<kStage>(words, rows, geo.row_words, walk_lds);
    int64_t i = (int64_t)blockIdx.x * kWalkThreads + threadIdx.x;
    if (i >= rows) return;
    if (done) {
        const int64_t g = row0 + i;
        if ((done[g >> 5] >> (g & 31)) & 1u) return;
    }
    margin[i] = margin[i] + t[walk_binned(t, nn, row, geo)].leaf_value;
}

__global__ void k_fill_u32(uint32_t *__restrict__ p, int64_t n, uint32_t v)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = v;
}

// Training rows whose node is known: entry i is row r = rows[i] (i when rows
// is NULL) in node pos[i].  When r is a row of the data, pos[i] a leaf of
// the tree and no earlier claim holds r, margin[r] receives the leaf and r
// is marked done; otherwise *bad counts the entry and r (if it is a row)
// is left to the traversal.
__global__ void k_margin_add_positions(const int32_t *__restrict__ rows, const int32_t *__restrict__ pos,
                                       int64_t n_pos, int64_t n_rows, const gbt_node *__restrict__ t, int32_t nn,
                                       float *__restrict__ margin, uint32_t *__restrict__ done,
                                       unsigned long long *__restrict__ bad)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n_pos) return;
    const int64_t r = rows ? rows[i] : i;
    const int32_t k = pos[i];
    const bool leaf = k >= 0 && k < nn && (t[k].flags & GBT_NODE_PRESENT) && (t[k].flags & GBT_NODE_LEAF);
    if (r < 0 || r >= n_rows || !leaf) {
        atomicAdd(bad, 1ull);
        return;
    }
    const uint32_t bit = 1u << (r & 31);
    if (atomicOr(&done[r >> 5], bit) & bit) {
        atomicAdd(bad, 1ull);  // the row appears twice
        return;
    }
    margin[r] = margin[r] + t[k].leaf_value;
}

static size_t walk_lds_bytes(const Geo &g) { return (size_t)kWalkThreads * (g.row_words + 1) * 4; }

// ------------------------------------------------------------ the iteration

// A tree whose kernels are queued: what the host needs to read its result.
struct TreePending {
    const void *res = nullptr;  // its pinned result (TreeResult)
    hipEvent_t done = nullptr;  // recorded after its last kernel, or NULL
    int64_t n = 0, R = 0;
    int32_t NN = 0, D = 0;
    bool mvs = false, stats = false;
    double key_lambda = 0.0;
    int32_t hist_launches = 0, hist_kind = 0, cols_bytes = 0;
    int64_t hist_bytes_fixed = 0;  // the root's part of the algorithmic bytes
    int64_t row_bytes_below = 0;   // per row built below the root
    int64_t node_hist_bytes = 0;   // per histogram built below the root
    double h2d = 0.0;
    std::chrono::steady_clock::time_point t_start;
};

// Queues one tree: gradients to the margin update, and the tree's copy into
// the pinned result res_h (res_d on the device), then `done` when not NULL.
// spec_prev: the MVS key exponent is guessed from the sampling state's last
// tree on the device (that tree is queued, and the host has not read it).
// reset_state: the tree's last kernel resets the sampling state for a next
// tree, which is then queued with state_ready (it skips state_init; both
// only for sampled trees on device pages).
static gbt_status train_tree_enqueue(gbt_ctx *c, const gbt_matrix *mx, const float *label, float *margin,
                                     const gbt_train_params *p, bool want_stats, void *res_h, void *res_d,
                                     hipEvent_t done, bool spec_prev, bool state_ready, bool reset_state,
                                     TreePending *pt)
{
    auto t_start = std::chrono::steady_clock::now();
    const int64_t n = mx->n_rows;
    const int32_t D = p->max_depth;
    const int32_t NN = (1 << (D + 1)) - 1;
    const bool host_pages = any_host_pages(mx);
    double h2d = 0.0;

    unsigned long long *upd = nullptr;  // zeroed with the tree's other counters
    if (want_stats) GBT_TRY(scratch_t(c, kScrUpd, kUpdWords, &upd));
    c->marks.clear();
    c->events_used = 0;
    int mark = timer_begin(c, kPhSample);
    float *gpair = nullptr;
    SampleState *st_ready = nullptr;
    const gbt_sample_params sp{p->f, p->mvs_lambda, p->seed, p->iteration, p->loss, p->sampler, p->goss_a};
    // MVS: the gradient pass sums the keys with the last tree's exponent, a
    // guess checked before the threshold is taken (the keys pass runs only
    // when it was wrong)
    const bool mvs = p->f < 1.0 && p->sampler == GBT_SAMPLE_MVS;
    int32_t e_spec = kNoKeySpec;
    if (mvs && !spec_prev && c->key_n_last == n && c->key_lambda_last == sample_lambda(sp)) e_spec = c->key_e_last;
    c->key_n_last = -1;  // set again when this tree has finished
    const int32_t *e_spec_at = nullptr;
    if (!host_pages) {
        GBT_TRY(scratch_t(c, kScrGpair, (size_t)std::max<int64_t>(n, 1) * 2, &gpair));
        if (p->f < 1.0) {
            // the gradient pass also folds the maximum of r for the sampling keys
            GBT_TRY(scratch_t(c, kScrState, 1, &st_ready));
            if (!state_ready) GBT_TRY(state_init(c, st_ready));
            if (mvs && spec_prev) e_spec_at = &st_ready->e_key_prev;
            GBT_TRY(gradients_rmax(c, p->loss, margin, label, n, gpair, sample_lambda(sp), st_ready, e_spec,
                                   e_spec_at));
        } else {
            GBT_TRY(launch_gradients(c, p->loss, margin, label, nullptr, n, gpair));
        }
    }
    Buffers bufs{c, false, {}};
    SampleOut so;
    GBT_TRY(sample_run(c, mx, gpair, margin, label, sp, bufs, &so, &h2d, st_ready, false,
                       st_ready != nullptr && (e_spec != kNoKeySpec || e_spec_at != nullptr)));
    timer_end(c, mark);
    const int64_t R = so.R;
    const int32_t *e_dev = &so.st->e_g;  // {e_g, e_h} on the device

    // ---- Alg. 1 on the sampled page, level by level.  Levels below the root
    // are planned on the device: no host round trip inside the tree.
    DevNode *nodes;
    int32_t *rows, *rows_tmp;
    float *leaf;
    gbt_split *splits_d;
    GBT_TRY(scratch_t(c, kScrNodes, (size_t)NN, &nodes));
    GBT_TRY(scratch_t(c, kScrLeaf, (size_t)NN, &leaf));
    GBT_TRY(scratch_t(c, kScrRows, (size_t)std::max<int64_t>(R, 1), &rows));
    GBT_TRY(scratch_t(c, kScrRowsTmp, (size_t)std::max<int64_t>(R, 1), &rows_tmp));
    // each slot's node, permuted with the rows
    int32_t *slot_node, *slot_tmp;
    GBT_TRY(scratch_t(c, kScrSlotA, (size_t)std::max<int64_t>(R, 1), &slot_node));
    GBT_TRY(scratch_t(c, kScrSlotB, (size_t)std::max<int64_t>(R, 1), &slot_tmp));
    const int32_t max_level_nodes =
        (int32_t)std::min<int64_t>((int64_t)1 << std::max(D - 1, 0), std::max<int64_t>(R, 1));
    GBT_TRY(scratch_t(c, kScrSplits, (size_t)max_level_nodes, &splits_d));
    const size_t hist_bytes = (size_t)max_level_nodes * (size_t)mx->total_bins * 16;
    int64_t *histA = nullptr, *histB = nullptr;
    if (D > 0) {
        GBT_TRY(scratch(c, kScrHistA, std::max<size_t>(hist_bytes, 16), (void **)&histA));
        GBT_TRY(scratch(c, kScrHistB, std::max<size_t>(hist_bytes, 16), (void **)&histB));
    }
    // plan buffers: two level lists, their counts, work items, reduce items, stats
    HistPlan hp;
    GBT_TRY(hist_plan(mx, R, c->hist_kernel, &hp));
    const std::vector<HistGroup> &groups = hp.groups;
    const int32_t G = (int32_t)groups.size();
    const int64_t twg = hp.target_wgs;
    // work items per group and level: one per workgroup slot (more only when
    // a level builds more than items / 2 nodes: then up to items plus the
    // node count)
    const int32_t items = (int32_t)std::max<int64_t>(1, twg / G);
    // the level plan scans its pass's chunk counts (at most items plus a
    // block of nodes) in 16 bits
    GBT_CHECK(items < (1 << 14), "%d work items per group", items);
    const int32_t max_work = items + max_level_nodes + 1;
    auto al = [](size_t b) { return (b + 255) / 256 * 256; };
    const size_t o_ev1 = al((size_t)max_level_nodes * sizeof(EvalNode));
    const size_t o_cnt = o_ev1 + o_ev1;
    // the root histogram: R rows in chunks, at most `items` - 1 per group
    const int64_t root_chunk =
        std::max<int64_t>(2048, (R + std::max(items - 1, 1) - 1) / std::max(items - 1, 1));
    const int32_t n_root = (int32_t)std::max<int64_t>(1, (R + root_chunk - 1) / root_chunk);
    const int32_t max_items = std::max(max_work, n_root);
    const size_t o_work = o_cnt + 256;
    const size_t o_red = o_work + al((size_t)max_items * sizeof(HistWork));
    const size_t plan_bytes = o_red + al((size_t)max_level_nodes * sizeof(HistReduce));
    char *plan;
    GBT_TRY(scratch_t(c, kScrPlan, plan_bytes, &plan));
    EvalNode *evA = (EvalNode *)plan, *evB = (EvalNode *)(plan + o_ev1);
    int32_t *cnt = (int32_t *)(plan + o_cnt);  // [0,1] level counts, [2] works, [3] reduces
    unsigned long long *stat = (unsigned long long *)(plan + o_cnt + 64);  // rows built, partials
    HistWork *work_d = (HistWork *)(plan + o_work);
    HistReduce *red_d = (HistReduce *)(plan + o_red);
    // the feature groups live with the matrix (uploaded once per kernel kind)
    // sparse pages: the slot table of the training page, and each feature's
    // group (stored after the groups)
    const bool use_tbl = hp.kind == kHistSparse && slot_table_fits(mx, G);
    const size_t fg_off = (std::max<size_t>(groups.size(), 1) * sizeof(HistGroup) + 15) / 16 * 16;
    if (mx->groups_kind != hp.kind) {
        // owned (and budgeted) by the matrix's context, like its other arrays
        std::vector<uint8_t> fg;
        if (use_tbl) {
            fg.assign((size_t)mx->m, 0);
            for (int32_t g = 0; g < G; ++g)
                for (int32_t f = groups[g].f0; f < groups[g].f1; ++f) fg[f] = (uint8_t)g;
        }
        const size_t gb = fg_off + fg.size();
        if (mx->groups_d) dev_free(mx->ctx, mx->groups_d, mx->groups_bytes);
        mx->groups_d = nullptr;
        mx->groups_kind = -1;
        GBT_TRY(dev_alloc(mx->ctx, gb, &mx->groups_d));
        mx->groups_bytes = gb;
        GBT_HIP(hipMemcpyAsync(mx->groups_d, groups.data(), groups.size() * sizeof(HistGroup),
                               hipMemcpyHostToDevice, c->stream));
        if (!fg.empty())
            GBT_HIP(hipMemcpyAsync((char *)mx->groups_d + fg_off, fg.data(), fg.size(), hipMemcpyHostToDevice,
                                   c->stream));
        GBT_HIP(hipStreamSynchronize(c->stream));
        mx->groups_kind = hp.kind;
    }
    const HistGroup *groups_d = (const HistGroup *)mx->groups_d;
    SlotTable stbl{nullptr, nullptr, nullptr, 0, 0, 0};
    if (use_tbl && D > 0 && R > 0) {
        const int32_t rs = slot_table_row_stride(G);
        const size_t col_off = ((size_t)R * rs + 255) / 256 * 256;
        uint8_t *tb;
        GBT_TRY(scratch_t(c, kScrSlotTbl, col_off + (size_t)R * G * sizeof(uint16_t), &tb));
        uint16_t *tc = (uint16_t *)(tb + col_off);
        GBT_TRY(sparse_slot_table(c, mx, groups_d, G, so.page, R, tb, tc));
        stbl = SlotTable{tb, tc, (const uint8_t *)mx->groups_d + fg_off, R, rs, 0};
    }
    // dense pages: the partition reads each row's split symbol from a column
    // copy of the training page, made once per tree (by the root histogram
    // pass for a sampled page of the plain kernel, else by split_columns;
    // once per matrix when the training page is the matrix's own device page)
    ColCopy cols;       // the copy the partition reads (cols.p NULL: none)
    ColCopy cols_root;  // the copy the root histogram pass writes
    const int32_t col_bytes = split_columns_fit(mx) ? split_columns_bytes(mx) : 0;
    if (D >= 2 && R > 0 && col_bytes &&
        scratch_fits(c, kScrCols, (size_t)mx->m * (size_t)R * (size_t)col_bytes)) {
        void *cd;
        GBT_TRY(scratch(c, kScrCols, (size_t)mx->m * (size_t)R * (size_t)col_bytes, &cd));
        const ColCopy cc{cd, R, col_bytes};
        const bool kept = so.alias && c->cols_uid == mx->uid && c->cols_page == so.page && c->cols_at == cd &&
                          c->cols_rows == R;
        if (!kept && !so.alias && hp.kind == kHistDense) {
            // a sampled page: the root pass of the plain kernel decodes every
            // symbol of every row anyway and writes the copy as it goes
            c->cols_uid = 0;
            cols_root = cc;
        } else if (!kept) {
            c->cols_uid = 0;
            GBT_TRY(split_columns(c, mx, so.page, R, cc));
            if (so.alias) {
                c->cols_uid = mx->uid;
                c->cols_page = so.page;
                c->cols_at = cd;
                c->cols_rows = R;
            }
        }
        cols = cc;
    }
    int64_t *partials = nullptr;
    GBT_TRY(scratch(c, kScrPartialsDev, (size_t)std::max(max_items, 1) * mx->total_bins * 16, (void **)&partials));
    // the root's slot arrays only for a tree without levels (whose leaves
    // may be added at the slots' rows); the root level's partition takes
    // slot i as row i of node 0 without reading them
    const int64_t n_slots = D == 0 ? R : 0;
    const int64_t n_init = std::max<int64_t>({(int64_t)NN, (int64_t)n_root, n_slots, (int64_t)kUpdCounters});
    k_tree_init<<<blocks(n_init), 256, 0, c->stream>>>(nodes, NN, so.st, R, evA, cnt, work_d, red_d, root_chunk,
                                                       n_root, rows, slot_node, n_slots, upd, stat);
    GBT_LAUNCHED();
    EvalParams ep{p->lambda, p->gamma, p->min_child_weight, 0, 0, e_dev};
    // features of at most 256 bins: each histogram pass ends with the fused
    // reduce + evaluate step, which evaluates the pass's nodes
    int32_t max_feature_bins = 0;
    for (int32_t f = 0; f < mx->m; ++f)
        max_feature_bins = std::max(max_feature_bins, mx->bin_ptr_h[f + 1] - mx->bin_ptr_h[f]);
    const bool fused = max_feature_bins <= 256;
    // the partition's flags pass makes each level's split choices from the
    // candidates (one wave per node and wave of slots) when a node has few
    // candidates and a level few nodes; otherwise a pass of its own does
    const bool choose = fused && mx->m <= 128 && max_level_nodes <= 4096;
    EvalCand *cand = nullptr;
    if (fused) GBT_TRY(scratch_t(c, kScrCand, (size_t)max_level_nodes * std::max(mx->m, 1), &cand));
    int32_t hist_launches = 0;
    int32_t *cntA = cnt, *cntB = cnt + 1;
    if (D > 0 && R > 0) {
        HistLaunch hl{hp.kind, groups_d, G, hp.max_groups_bins, work_d, nullptr, n_root, red_d, nullptr,
                      fused ? 0 : 1, partials, stbl.row, stbl.row_stride};
        hl.cols = cols_root;  // the root's work items cover rows [0, R) once per group
        GBT_TRY(hist_launch_device(c, mx, so.page, so.q, nullptr, hl, nullptr, histA, upd));
        ++hist_launches;
        if (fused) {
            mark = timer_begin(c, kPhHistAux);
            GBT_TRY(reduce_eval_impl(c, mx, partials, red_d, nullptr, 1, nullptr, histA, evA, ep, cand));
            if (!choose) GBT_TRY(eval_reduce_impl(c, mx, cand, mx->m, evA, 1, cntA, splits_d, nodes));
            timer_end(c, mark);
        }
    }
    // the walk's compact tree and the leaf values: made by the last level's
    // plan (by k_leaves when there is no level or no row)
    uint2 *compact;
    GBT_TRY(scratch_t(c, kScrCompact, (size_t)NN, &compact));
    const bool leaves_in_plan = D > 0 && R > 0;
    // the rows' final slots give their leaves (below) only on sparse pages
    // that are the data's own page; otherwise nothing reads the last
    // level's row order and its partition only counts
    const bool final_order = so.alias && mx->sparse;
    for (int32_t d = 0; d < D; ++d) {
        const int32_t maxn = (int32_t)std::min<int64_t>((int64_t)1 << d, max_level_nodes);
        mark = timer_begin(c, kPhSplit);
        if (!fused && R > 0) GBT_TRY(eval_impl(c, mx, histA, evA, maxn, ep, splits_d, cntA, nodes));
        const LevelChoice lc{cand, mx->m, (int32_t)((1u << d) - 1), (int32_t)((2u << d) - 1)};
        const bool plan_next = d + 1 < D && R > 0;
        // the partition's second kernel also plans the next level (and
        // after the last level makes the leaves)
        const bool last = d + 1 == D;
        PlanArgs pa{evA, cntA, plan_next ? 1 : 0, items, evB, cntB, work_d, cnt + 2, red_d, cnt + 3, stat};
        if (last) pa.lv = LeafArgs{leaf, compact, e_dev, p->lambda, p->eta, NN, 0};
        GBT_TRY(partition_rev_impl(c, mx, so.page, rows, R, slot_node, slot_tmp, nodes, rows_tmp,
                                   choose ? &lc : nullptr, stbl.row ? &stbl : nullptr, cols, pa,
                                   !last || final_order, d == 0));
        std::swap(rows, rows_tmp);
        std::swap(slot_node, slot_tmp);
        timer_end(c, mark);
        if (plan_next) {
            HistLaunch hl{hp.kind, groups_d, G, hp.max_groups_bins, work_d, cnt + 2, max_work, red_d, cnt + 3,
                          fused ? 0 : maxn, partials, stbl.row, stbl.row_stride};
            GBT_TRY(hist_launch_device(c, mx, so.page, so.q, rows, hl, histA, histB, upd));
            ++hist_launches;
            if (fused) {
                // the next level: at most 2 maxn nodes, in evB
                const int32_t nxt = (int32_t)std::min<int64_t>(2 * (int64_t)maxn, max_level_nodes);
                mark = timer_begin(c, kPhHistAux);
                // the deepest evaluated level's histograms are nobody's parents
                GBT_TRY(reduce_eval_impl(c, mx, partials, red_d, cnt + 3, maxn, histA, d + 2 < D ? histB : nullptr,
                                         evB, ep, cand));
                if (!choose) GBT_TRY(eval_reduce_impl(c, mx, cand, mx->m, evB, nxt, cntB, splits_d, nodes));
                timer_end(c, mark);
            }
            std::swap(histA, histB);
            std::swap(evA, evB);
            std::swap(cntA, cntB);
        }
    }
    // ---- leaves and the margin update of all n rows (Eq. 1)
    mark = timer_begin(c, kPhMargin);
    if (!leaves_in_plan) {
        k_leaves<<<blocks(NN), 256, 0, c->stream>>>(nodes, NN, e_dev, p->lambda, p->eta, leaf, compact);
        GBT_LAUNCHED();
    }
    // the tree and the counters: written by the device into pinned memory,
    // read after the one synchronization of the call; with the dense walk,
    // by two more blocks of its first launch
    const FinalizeArgs fa{nodes, NN, 0, leaf, mx->cut_ptr_d, mx->cut_values_d, so.st, upd, stat,
                          (TreeResult *)res_d, reset_state ? so.st : nullptr};
    bool finalized = false;
    // the rows' final slots give their leaves when every row trained; on
    // dense pages the walk of the page in row order is cheaper than adding
    // into the margins at the slots' (scattered) rows
    if (final_order) {
        if (n) {
            k_margin_slots<<<blocks(n), 256, 0, c->stream>>>(margin, rows, slot_node, leaf, n);
            GBT_LAUNCHED();
        }
    } else {
        Geo geo = geo_of(mx);
        GBT_TRY(for_each_chunk(
            c, mx,
            [&](const uint32_t *words, int64_t row0, int64_t rows_n) -> gbt_status {
                const size_t lds_bytes = (size_t)NN * 12 + (size_t)kWalkTileRows * (geo.row_words + 1) * 4;
                const int q4 = geo.row_words / 4;
                // one block per tile: independent blocks hide the page's
                // latency better than a smaller grid that prefetches
                if (q4 <= 8 && NN <= kWalkLdsNodes && lds_bytes <= 64 * 1024) {
                    int64_t tiles = (rows_n + kWalkTileRows - 1) / kWalkTileRows;
                    unsigned grid = (unsigned)tiles;
                    const int32_t fin = finalized ? 0 : (int32_t)blocks(NN);
                    launch_walk_pf(c, q4, grid, lds_bytes, words, rows_n, geo, compact, leaf, NN, margin + row0,
                                   fin, fa);
                    finalized = true;
                } else if (geo.row_words <= kWalkMaxWords && NN <= kWalkLdsNodes && lds_bytes <= 64 * 1024) {
                    int64_t tiles = (rows_n + kWalkTileRows - 1) / kWalkTileRows;
                    unsigned grid = (unsigned)std::min<int64_t>(tiles, 4 * kCUs);
                    k_margin_walk_lds<<<grid, kWalkTileRows, lds_bytes, c->stream>>>(words, rows_n, geo, compact,
                                                                                     leaf, NN, margin + row0);
                } else if (geo.row_words <= kWalkMaxWords)
                    k_margin_walk<true><<<blocks(rows_n), kWalkThreads, walk_lds_bytes(geo), c->stream>>>(
                        words, rows_n, geo, nodes, leaf, margin + row0);
                else
                    k_margin_walk<false><<<blocks(rows_n), kWalkThreads, 0, c->stream>>>(
                        words, rows_n, geo, nodes, leaf, margin + row0);
                GBT_LAUNCHED();
                return GBT_OK;
            },
            &h2d));
    }
    timer_end(c, mark);
    if (!finalized) {
        k_finalize<<<blocks(NN), 256, 0, c->stream>>>(fa);
        GBT_LAUNCHED();
    }
    if (done) GBT_HIP(hipEventRecord(done, c->stream));
    // algorithmic bytes of the histogram passes: the packed symbols of each
    // row, its 16-byte fixed-point pair, its 4-byte row id below the root,
    // one write of every built node's histogram (the chunk partials are not
    // counted), and the column copy when the root pass writes it (1 or 2
    // bytes per symbol)
    const int64_t wbytes = 4 * (((int64_t)mx->stride * mx->w + 31) / 32);
    const int64_t root_built = (D > 0 && R > 0) ? 1 : 0;
    pt->res = res_h;
    pt->done = done;
    pt->n = n;
    pt->R = R;
    pt->NN = NN;
    pt->D = D;
    pt->mvs = mvs;
    pt->stats = want_stats;
    pt->key_lambda = sample_lambda(sp);
    pt->hist_launches = hist_launches;
    pt->hist_kind = hp.kind == kHistRot ? GBT_HIST_ROTATED : (hp.kind == kHistDense ? GBT_HIST_PLAIN : 0);
    pt->cols_bytes = cols_root.bytes;
    pt->hist_bytes_fixed = (D > 0 ? R : 0) * (wbytes + 16) + root_built * mx->total_bins * 16 +
                           (int64_t)cols_root.bytes * mx->m * R;
    pt->row_bytes_below = wbytes + 20;
    pt->node_hist_bytes = mx->total_bins * 16;
    pt->h2d = h2d;
    pt->t_start = t_start;
    return GBT_OK;
}

// Reads a queued tree's result into `tree` (and `stats`, when the tree was
// queued with them); the caller has waited for its last kernels.
static gbt_status train_tree_finish(gbt_ctx *c, const TreePending &pt, gbt_tree *tree, gbt_tree_stats *stats)
{
    const TreeResult *res = (const TreeResult *)pt.res;
    if (res->bad) return set_error(GBT_E_INVALID, "sampling failed (state flags %u)", res->bad);
    if (pt.mvs) {
        c->key_e_last = res->e_key;
        c->key_n_last = pt.n;
        c->key_lambda_last = pt.key_lambda;
    }
    tree->max_depth = pt.D;
    tree->exp_g = res->e_g;
    tree->exp_h = res->e_h;
    memcpy(tree->nodes, res->nodes, (size_t)pt.NN * sizeof(gbt_node));
    double ms[kPhCount] = {0.0};
    timer_collect(c, ms);
    if (stats && pt.stats) {
        memset(stats, 0, sizeof(*stats));
        stats->n_sampled = pt.R;
        stats->threshold = res->T;
        stats->exp_key = res->e_key;
        stats->hist_updates = (int64_t)res->updates;
        stats->hist_launches = pt.hist_launches;
        stats->hist_rows = (pt.D > 0 ? pt.R : 0) + (int64_t)res->rows_built;
        stats->hist_bytes = pt.hist_bytes_fixed + (int64_t)res->rows_built * pt.row_bytes_below +
                            (int64_t)res->built * pt.node_hist_bytes;
        stats->ms_sample = ms[kPhSample];
        stats->ms_hist = ms[kPhHist];
        stats->ms_hist_aux = ms[kPhHistAux];
        stats->ms_split = ms[kPhSplit];
        stats->ms_margin = ms[kPhMargin];
        stats->h2d_bytes = pt.h2d;
        stats->hist_kernel = pt.hist_kind;
        stats->hist_cols = pt.cols_bytes;
        stats->ms_total =
            std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - pt.t_start).count();
    }
    return GBT_OK;
}

// Bytes of one tree's pinned result (a multiple of 256).
static size_t tree_result_bytes(int32_t NN)
{
    return (sizeof(TreeResult) + (size_t)NN * sizeof(gbt_node) + 255) / 256 * 256;
}

static gbt_status train_tree_impl(gbt_ctx *c, const gbt_matrix *mx, const float *label, float *margin,
                                  const gbt_train_params *p, gbt_tree *tree, gbt_tree_stats *stats)
{
    void *rh, *rd;
    GBT_TRY(tree_io(c, tree_result_bytes((1 << (p->max_depth + 1)) - 1), &rh, &rd));
    TreePending pt;
    GBT_TRY(train_tree_enqueue(c, mx, label, margin, p, stats != nullptr, rh, rd, nullptr, false, false, false,
                               &pt));
    GBT_HIP(hipStreamSynchronize(c->stream));
    return train_tree_finish(c, pt, tree, stats);
}

static gbt_status upload_trees(gbt_ctx *c, const gbt_tree *trees, int32_t n_trees, gbt_node **nodes_d,
                               int64_t **offs_d)
{
    std::vector<int64_t> offs(n_trees + 1, 0);
    for (int32_t t = 0; t < n_trees; ++t) {
        GBT_CHECK(trees[t].nodes && trees[t].n_nodes > 0, "tree %d has no nodes", t);
        offs[t + 1] = offs[t] + trees[t].n_nodes;
    }
    size_t o_off = ((size_t)offs[n_trees] * sizeof(gbt_node) + 255) / 256 * 256;
    char *buf;
    GBT_TRY(scratch_t(c, kScrTrees, o_off + (n_trees + 1) * 8, &buf));
    std::vector<char> h(o_off + (n_trees + 1) * 8);
    for (int32_t t = 0; t < n_trees; ++t)
        memcpy(h.data() + offs[t] * sizeof(gbt_node), trees[t].nodes, trees[t].n_nodes * sizeof(gbt_node));
    memcpy(h.data() + o_off, offs.data(), (n_trees + 1) * 8);
    GBT_HIP(hipMemcpyAsync(buf, h.data(), h.size(), hipMemcpyHostToDevice, c->stream));
    *nodes_d = (gbt_node *)buf;
    *offs_d = (int64_t *)(buf + o_off);
    return GBT_OK;
}

}  // namespace gbt

using namespace gbt;

struct gbt_sampled {
    gbt_ctx *ctx = nullptr;
    Buffers bufs{nullptr, true, {}};
    SampleOut out;
    int32_t row_words = 0;
};

extern "C" {

gbt_status gbt_gradients(gbt_ctx *c, int32_t loss, const float *margin_d, const float *label_d,
                         const float *weight_d, int64_t n, float *gpair_d)
{
    GBT_CHECK(c, "ctx is NULL");
    GBT_CHECK(n >= 0, "n < 0");
    GBT_CHECK(loss == GBT_LOSS_LOGISTIC || loss == GBT_LOSS_SQUARED, "unknown loss %d", loss);
    GBT_CHECK(n == 0 || (margin_d && label_d && gpair_d), "gbt_gradients: NULL array");
    GBT_TRY(set_device(c));
    GBT_TRY(launch_gradients(c, loss, margin_d, label_d, weight_d, n, gpair_d));
    GBT_HIP(hipStreamSynchronize(c->stream));
    return GBT_OK;
}

gbt_status gbt_mvs_lambda_estimate(gbt_ctx *c, int32_t loss, const float *margin_d, const float *label_d, int64_t n,
                                   double *lambda_out)
{
    GBT_CHECK(c && lambda_out, "gbt_mvs_lambda_estimate: NULL argument");
    GBT_CHECK(n >= 0, "n < 0");
    GBT_CHECK(loss == GBT_LOSS_LOGISTIC || loss == GBT_LOSS_SQUARED, "unknown loss %d", loss);
    GBT_CHECK(n == 0 || (margin_d && label_d), "gbt_mvs_lambda_estimate: NULL array");
    *lambda_out = 0.0;
    if (n == 0) return GBT_OK;
    GBT_TRY(set_device(c));
    // every row's pair in its exact fixed point over the n rows; two passes
    // fold the maxima, then the integer sums, into the state (no per-row
    // buffer, so the call fits any budget that holds the state)
    SampleState *st;
    GBT_TRY(scratch_t(c, kScrState, 1, &st));
    GBT_TRY(state_init(c, st));
    GBT_TRY(lambda_sums(c, loss, margin_d, label_d, n, st));
    SampleState hst;
    GBT_HIP(hipMemcpyAsync(&hst, st, sizeof(SampleState), hipMemcpyDeviceToHost, c->stream));
    GBT_HIP(hipStreamSynchronize(c->stream));
    if (hst.bad) return set_error(GBT_E_INVALID, "gradient sums failed (state flags %u)", hst.bad);
    const long long G = (long long)fold_sum(hst.root_g), H = (long long)fold_sum(hst.root_h);
    if (H != 0) {
        const double w0 = -std::ldexp((double)G, -hst.e_g) / std::ldexp((double)H, -hst.e_h);
        *lambda_out = w0 * w0;
    }
    return GBT_OK;
}

gbt_status gbt_sample(gbt_ctx *c, const gbt_matrix *data, const float *gpair_d, const float *margin_d,
                      const float *label_d, const gbt_sample_params *sp, gbt_sampled **out)
{
    GBT_CHECK(c && data && sp && out, "gbt_sample: NULL argument");
    *out = nullptr;
    GBT_CHECK(sp->loss == GBT_LOSS_LOGISTIC || sp->loss == GBT_LOSS_SQUARED || gpair_d, "unknown loss");
    GBT_TRY(set_device(c));
    auto *s = new gbt_sampled();
    s->ctx = c;
    s->bufs.c = c;
    s->row_words = data->row_words;
    gbt_status st = sample_run(c, data, gpair_d, margin_d, label_d, *sp, s->bufs, &s->out, nullptr);
    if (st == GBT_OK) {
        hipError_t e = hipStreamSynchronize(c->stream);
        if (e != hipSuccess) st = hip_error(e, "sync", __FILE__, __LINE__);
    }
    if (st != GBT_OK) {
        (void)hipStreamSynchronize(c->stream);
        s->bufs.release();
        delete s;
        return st;
    }
    *out = s;
    return GBT_OK;
}

gbt_status gbt_sampled_info_get(const gbt_sampled *s, gbt_sampled_info *info)
{
    GBT_CHECK(s && info, "gbt_sampled_info_get: NULL argument");
    info->n_sampled = s->out.R;
    info->threshold = s->out.T;
    info->target = s->out.K;
    info->exp_key = s->out.e_key;
    info->exp_g = s->out.e_g;
    info->exp_h = s->out.e_h;
    info->is_alias = s->out.alias ? 1 : 0;
    info->page_d = s->out.page;
    info->rows_d = s->out.sel;
    info->gpair_d = s->out.gw;
    info->gpair_fx_d = s->out.q;
    return GBT_OK;
}

gbt_status gbt_sampled_free(gbt_sampled *s)
{
    if (!s) return GBT_OK;
    (void)hipSetDevice(s->ctx->device);
    (void)hipStreamSynchronize(s->ctx->stream);
    s->bufs.release();
    delete s;
    return GBT_OK;
}

// ------------------------------------------------------------ Alg. 6
// The naive out-of-core construction (Sec. 3.3), a measured negative
// baseline: every row trains and every level streams every page once.  A
// level's pass moves each row to its node (the row's node id is kept for all
// n rows), groups the chunk's rows by the level's nodes and builds every
// node's histogram from them (both children: no page stays resident, so a
// parent's histogram cannot be reused across passes).  One last pass moves
// the rows to the leaves, whose ids give the margin update.
constexpr int32_t kNaiveMaxDepth = 11;  // at most 2048 nodes per level (LDS counts)
constexpr int32_t kNaiveSlots = 1 << kNaiveMaxDepth;

// Route the chunk's rows one level down (when `move`) and count them per
// node slot of the current level (slot_of: heap id -> slot, -1 outside it).
__global__ void __launch_bounds__(256)
    k_naive_route(const uint32_t *__restrict__ words, int64_t rows, int64_t row0, Geo geo,
                  const DevNode *__restrict__ nodes, int32_t *__restrict__ position,
                  const int32_t *__restrict__ slot_of, int32_t n_slots, int32_t move, uint32_t *__restrict__ cnt)
{
    __shared__ uint32_t lc[kNaiveSlots];
    for (int32_t s = threadIdx.x; s < n_slots; s += 256) lc[s] = 0;
    __syncthreads();
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < rows) {
        int32_t p = position[row0 + i];
        if (move) {
            const int4 rec = *(const int4 *)&nodes[p].split;
            if (rec.x) {
                const int32_t b = row_feature_bin(words + i * geo.row_words, geo, rec.y);
                const bool left = b < 0 ? rec.w != 0 : b < rec.z;
                p = left ? nodes[p].left_child : nodes[p].right_child;
                position[row0 + i] = p;
            }
        }
        const int32_t s = slot_of[p];
        if (s >= 0) atomicAdd(&lc[s], 1u);
    }
    __syncthreads();
    for (int32_t s = threadIdx.x; s < n_slots; s += 256)
        if (lc[s]) atomicAdd(&cnt[s], lc[s]);
}

// The chunk's rows grouped by slot: a block ranks its rows per slot in LDS,
// reserves each slot's range with one atomic, and writes the local row ids.
__global__ void __launch_bounds__(256)
    k_naive_group(int64_t rows, int64_t row0, const int32_t *__restrict__ position,
                  const int32_t *__restrict__ slot_of, int32_t n_slots, uint32_t *__restrict__ cursor,
                  int32_t *__restrict__ grouped)
{
    __shared__ uint32_t lc[kNaiveSlots];
    __shared__ uint32_t base[kNaiveSlots];
    for (int32_t s = threadIdx.x; s < n_slots; s += 256) lc[s] = 0;
    __syncthreads();
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    int32_t s = -1;
    uint32_t rank = 0;
    if (i < rows) {
        s = slot_of[position[row0 + i]];
        if (s >= 0) rank = atomicAdd(&lc[s], 1u);
    }
    __syncthreads();
    for (int32_t t = threadIdx.x; t < n_slots; t += 256) base[t] = lc[t] ? atomicAdd(&cursor[t], lc[t]) : 0u;
    __syncthreads();
    if (s >= 0) grouped[base[s] + rank] = (int32_t)i;
}

// hist[slot] += part[slot] for the listed slots.
__global__ void k_naive_accumulate(longlong2 *__restrict__ hist, const longlong2 *__restrict__ part,
                                   const int32_t *__restrict__ slots, int32_t n, int64_t tb)
{
    const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= tb) return;
    const int64_t s = slots[blockIdx.y];
    longlong2 h = hist[s * tb + b];
    const longlong2 v = part[s * tb + b];
    h.x += v.x;
    h.y += v.y;
    hist[s * tb + b] = h;
}

// margin[r] += leaf of the row's final node.
__global__ void k_naive_margin(float *__restrict__ margin, const int32_t *__restrict__ position,
                               const float *__restrict__ leaf, int64_t n)
{
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r < n) margin[r] += leaf[position[r]];
}

__global__ void k_naive_zero(unsigned long long *__restrict__ p, int64_t n)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0ull;
}

__global__ void k_fill_i32(int32_t *__restrict__ p, int64_t n, int32_t v)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = v;
}

static gbt_status train_tree_naive_impl(gbt_ctx *c, const gbt_matrix *mx, const float *label, float *margin,
                                        const gbt_train_params *p, gbt_tree *tree, gbt_tree_stats *stats)
{
    const auto t_start = std::chrono::steady_clock::now();
    const int64_t n = mx->n_rows;
    const int32_t D = p->max_depth;
    const int32_t NN = (1 << (D + 1)) - 1;
    const int64_t tb = mx->total_bins;
    double h2d = 0.0;
    c->marks.clear();
    c->events_used = 0;
    // gradients and their exact fixed point over all n rows (no sampling)
    int mark = timer_begin(c, kPhSample);
    float *gpair;
    double *gw;
    int64_t *q;
    SampleState *st;
    GBT_TRY(scratch_t(c, kScrGpair, (size_t)std::max<int64_t>(n, 1) * 2, &gpair));
    GBT_TRY(scratch_t(c, kScrGw, (size_t)std::max<int64_t>(n, 1) * 2, &gw));
    GBT_TRY(scratch_t(c, kScrQ, (size_t)std::max<int64_t>(n, 1) * 2, &q));
    GBT_TRY(scratch_t(c, kScrState, 1, &st));
    GBT_TRY(state_init(c, st));
    GBT_TRY(launch_gradients(c, p->loss, margin, label, nullptr, n, gpair));
    GBT_TRY(gw_all(c, gpair, n, gw));
    GBT_TRY(fixed_point(c, gw, n, st, q, false));
    SampleState hst;
    GBT_HIP(hipMemcpyAsync(&hst, st, sizeof(SampleState), hipMemcpyDeviceToHost, c->stream));
    GBT_HIP(hipStreamSynchronize(c->stream));
    timer_end(c, mark);
    // the node table on the host (uploaded each level), each row's node
    std::vector<DevNode> hn((size_t)NN);
    for (int32_t i = 0; i < NN; ++i) {
        memset(&hn[i], 0, sizeof(DevNode));
        hn[i].left_child = 2 * i + 1;
        hn[i].right_child = 2 * i + 2;
    }
    hn[0].present = 1;
    hn[0].sum_g = (long long)fold_sum(hst.root_g);
    hn[0].sum_h = (long long)fold_sum(hst.root_h);
    hn[0].end = n;
    DevNode *nodes;
    int32_t *position, *slot_of, *grouped;
    uint32_t *cnt;
    gbt_split *splits_d;
    EvalNode *ev_d;
    int32_t *slots_d;
    const int32_t max_level = 1 << D;
    int64_t chunk_rows = 1;  // the largest chunk for_each_chunk passes
    for (const auto &pg : mx->pages)
        chunk_rows = std::max(chunk_rows, pg.streamed() ? std::min(pg.rows, c->stream_chunk_rows) : pg.rows);
    GBT_TRY(scratch_t(c, kScrNodes, (size_t)NN, &nodes));
    GBT_TRY(scratch_t(c, kScrPosition, (size_t)std::max<int64_t>(n, 1), &position));
    GBT_TRY(scratch_t(c, kScrSlotNode, (size_t)NN, &slot_of));
    GBT_TRY(scratch_t(c, kScrRows, (size_t)chunk_rows, &grouped));
    GBT_TRY(scratch_t(c, kScrScan, (size_t)2 * max_level, &cnt));
    GBT_TRY(scratch_t(c, kScrSplits, (size_t)max_level, &splits_d));
    GBT_TRY(scratch_t(c, kScrEvalNodes, (size_t)max_level, &ev_d));
    GBT_TRY(scratch_t(c, kScrPlan, (size_t)max_level, &slots_d));
    int64_t *hist = nullptr, *part = nullptr;
    if (D > 0) {
        GBT_TRY(scratch_t(c, kScrHistA, (size_t)max_level * tb * 2, &hist));
        GBT_TRY(scratch_t(c, kScrHistB, (size_t)max_level * tb * 2, &part));
    }
    if (n) {
        k_fill_i32<<<blocks(n), 256, 0, c->stream>>>(position, n, 0);
        GBT_LAUNCHED();
    }
    const Geo geo = geo_of(mx);
    const EvalParams ep{p->lambda, p->gamma, p->min_child_weight, 0, 0, &st->e_g};
    // the histogram launches' counters: updates on the device, rows and
    // algorithmic bytes on the host
    unsigned long long *upd;
    GBT_TRY(scratch_t(c, kScrUpd, kUpdWords, &upd));
    k_naive_zero<<<blocks(kUpdWords), 256, 0, c->stream>>>(upd, kUpdWords);
    GBT_LAUNCHED();
    gbt_tree_stats hs;
    memset(&hs, 0, sizeof(hs));
    int64_t kind_rows[3] = {0, 0, 0};  // rows built by the sparse, plain and rotated kernels
    std::vector<int32_t> level{0}, so((size_t)NN, -1);
    std::vector<uint32_t> hcnt;
    for (int32_t d = 0; d <= D && n > 0; ++d) {
        const int32_t L = (int32_t)level.size();
        if (L == 0) break;
        const bool build = d < D;
        std::fill(so.begin(), so.end(), -1);
        for (int32_t s = 0; s < L; ++s) so[level[s]] = s;
        GBT_HIP(hipMemcpyAsync(nodes, hn.data(), (size_t)NN * sizeof(DevNode), hipMemcpyHostToDevice, c->stream));
        GBT_HIP(hipMemcpyAsync(slot_of, so.data(), (size_t)NN * 4, hipMemcpyHostToDevice, c->stream));
        if (build) {
            k_naive_zero<<<blocks((int64_t)L * tb * 2), 256, 0, c->stream>>>((unsigned long long *)hist, (int64_t)L * tb * 2);
            GBT_LAUNCHED();
        }
        std::vector<uint64_t> total((size_t)L, 0);
        GBT_TRY(for_each_chunk(
            c, mx,
            [&](const uint32_t *words, int64_t row0, int64_t rows) -> gbt_status {
                k_naive_zero<<<blocks(L), 256, 0, c->stream>>>((unsigned long long *)cnt, (L + 1) / 2);
                GBT_LAUNCHED();
                k_naive_route<<<(unsigned)((rows + 255) / 256), 256, 0, c->stream>>>(
                    words, rows, row0, geo, nodes, position, slot_of, L, d > 0 ? 1 : 0, cnt);
                GBT_LAUNCHED();
                hcnt.assign((size_t)L, 0);
                GBT_HIP(hipMemcpyAsync(hcnt.data(), cnt, (size_t)L * 4, hipMemcpyDeviceToHost, c->stream));
                GBT_HIP(hipStreamSynchronize(c->stream));
                for (int32_t s = 0; s < L; ++s) total[s] += hcnt[s];
                if (!build) return GBT_OK;
                // group the chunk's rows by slot and build their histograms
                std::vector<uint32_t> cur((size_t)L);
                std::vector<gbt_seg> segs;
                std::vector<int32_t> built;
                uint32_t off = 0;
                for (int32_t s = 0; s < L; ++s) {
                    cur[s] = off;
                    if (hcnt[s]) {
                        segs.push_back(gbt_seg{s, 0, off, off + hcnt[s]});
                        built.push_back(s);
                    }
                    off += hcnt[s];
                }
                if (segs.empty()) return GBT_OK;
                HistPlan hpk;
                GBT_TRY(hist_plan(mx, off, c->hist_kernel, &hpk));
                kind_rows[hpk.kind == kHistRot ? 2 : (hpk.kind == kHistDense ? 1 : 0)] += off;
                GBT_HIP(hipMemcpyAsync(cnt, cur.data(), (size_t)L * 4, hipMemcpyHostToDevice, c->stream));
                k_naive_group<<<(unsigned)((rows + 255) / 256), 256, 0, c->stream>>>(rows, row0, position, slot_of,
                                                                                      L, cnt, grouped);
                GBT_LAUNCHED();
                GBT_TRY(build_hist_impl(c, mx, words, q + 2 * row0, grouped, segs.data(), (int32_t)segs.size(),
                                        nullptr, 0, nullptr, part, &hs));
                GBT_HIP(hipMemcpyAsync(slots_d, built.data(), built.size() * 4, hipMemcpyHostToDevice, c->stream));
                dim3 g((unsigned)((tb + 255) / 256), (unsigned)built.size());
                k_naive_accumulate<<<g, 256, 0, c->stream>>>((longlong2 *)hist, (const longlong2 *)part, slots_d,
                                                             (int32_t)built.size(), tb);
                GBT_LAUNCHED();
                // the host vectors above are read by the copies before this
                // chunk returns
                GBT_HIP(hipStreamSynchronize(c->stream));
                return GBT_OK;
            },
            &h2d));
        for (int32_t s = 0; s < L; ++s) {
            hn[level[s]].begin = 0;
            hn[level[s]].end = (int64_t)total[s];
        }
        if (!build) break;
        // Eq. 8 for every node of the level; the split records land in the
        // device node table, then come back to the host
        mark = timer_begin(c, kPhSplit);
        std::vector<EvalNode> ev((size_t)L);
        for (int32_t s = 0; s < L; ++s) ev[s] = EvalNode{hn[level[s]].sum_g, hn[level[s]].sum_h, s, level[s]};
        GBT_HIP(hipMemcpyAsync(ev_d, ev.data(), (size_t)L * sizeof(EvalNode), hipMemcpyHostToDevice, c->stream));
        GBT_HIP(hipMemcpyAsync(nodes, hn.data(), (size_t)NN * sizeof(DevNode), hipMemcpyHostToDevice, c->stream));
        GBT_TRY(eval_impl(c, mx, hist, ev_d, L, ep, splits_d, nullptr, nodes));
        GBT_HIP(hipMemcpyAsync(hn.data(), nodes, (size_t)NN * sizeof(DevNode), hipMemcpyDeviceToHost, c->stream));
        GBT_HIP(hipStreamSynchronize(c->stream));
        timer_end(c, mark);
        std::vector<int32_t> next;
        for (int32_t s = 0; s < L; ++s) {
            const DevNode &x = hn[level[s]];
            if (!x.split) continue;
            DevNode &l = hn[x.left_child], &r = hn[x.right_child];
            l.present = r.present = 1;
            l.sum_g = x.left_g;
            l.sum_h = x.left_h;
            r.sum_g = x.right_g;
            r.sum_h = x.right_h;
            next.push_back(x.left_child);
            next.push_back(x.right_child);
        }
        // the children's rows move in the next pass
        level.swap(next);
        if (level.empty()) break;
    }
    // ---- leaves, the margin update of all n rows, the public tree
    mark = timer_begin(c, kPhMargin);
    GBT_HIP(hipMemcpyAsync(nodes, hn.data(), (size_t)NN * sizeof(DevNode), hipMemcpyHostToDevice, c->stream));
    float *leaf;
    uint2 *compact;
    GBT_TRY(scratch_t(c, kScrLeaf, (size_t)NN, &leaf));
    GBT_TRY(scratch_t(c, kScrCompact, (size_t)NN, &compact));
    k_leaves<<<blocks(NN), 256, 0, c->stream>>>(nodes, NN, &st->e_g, p->lambda, p->eta, leaf, compact);
    GBT_LAUNCHED();
    if (n) {
        k_naive_margin<<<blocks(n), 256, 0, c->stream>>>(margin, position, leaf, n);
        GBT_LAUNCHED();
    }
    timer_end(c, mark);
    unsigned long long *stat;
    GBT_TRY(scratch_t(c, kScrWork, 2, &stat));
    k_naive_zero<<<1, 256, 0, c->stream>>>(stat, 2);
    GBT_LAUNCHED();
    void *hio, *hio_d;
    GBT_TRY(host_io(c, sizeof(TreeResult) + (size_t)NN * sizeof(gbt_node), &hio, &hio_d));
    k_finalize<<<blocks(NN), 256, 0, c->stream>>>(
        FinalizeArgs{nodes, NN, 0, leaf, mx->cut_ptr_d, mx->cut_values_d, st, upd, stat, (TreeResult *)hio_d,
                     nullptr});
    GBT_LAUNCHED();
    GBT_HIP(hipStreamSynchronize(c->stream));
    const TreeResult *res = (const TreeResult *)hio;
    tree->exp_g = res->e_g;
    tree->exp_h = res->e_h;
    memcpy(tree->nodes, res->nodes, (size_t)NN * sizeof(gbt_node));
    double ms[kPhCount] = {0.0};
    timer_collect(c, ms);
    if (stats) {
        stats->n_sampled = n;
        stats->hist_launches = hs.hist_launches;
        stats->hist_rows = hs.hist_rows;
        stats->hist_bytes = hs.hist_bytes;
        stats->hist_updates = (int64_t)res->updates;
        // the kernel that built the most rows
        stats->hist_kernel = mx->sparse ? 0
                             : (kind_rows[2] >= kind_rows[1] ? GBT_HIST_ROTATED : GBT_HIST_PLAIN);
        stats->h2d_bytes = (int64_t)h2d;
        stats->ms_sample = ms[kPhSample];
        stats->ms_hist = ms[kPhHist];
        stats->ms_split = ms[kPhSplit];
        stats->ms_margin = ms[kPhMargin];
        stats->ms_total =
            std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t_start).count();
    }
    return GBT_OK;
}

gbt_status gbt_train_tree_naive(gbt_ctx *c, const gbt_matrix *data, const float *label_d, float *margin_d,
                                const gbt_train_params *p, gbt_tree *tree, gbt_tree_stats *stats)
{
    GBT_CHECK(c && data && p && tree && tree->nodes, "gbt_train_tree_naive: NULL argument");
    GBT_CHECK(data->n_rows == 0 || (label_d && margin_d), "gbt_train_tree_naive: NULL labels/margins");
    GBT_TRY(hist_check_feature_bins(data));
    GBT_CHECK(p->max_depth >= 0 && p->max_depth <= kNaiveMaxDepth, "max_depth %d outside [0, %d]", p->max_depth,
              kNaiveMaxDepth);
    GBT_CHECK(p->f == 1.0, "the naive construction trains every row (f = 1, got %g)", p->f);
    GBT_CHECK(p->loss == GBT_LOSS_LOGISTIC || p->loss == GBT_LOSS_SQUARED, "unknown loss %d", p->loss);
    GBT_CHECK(data->n_rows < ((int64_t)1 << 31) - 1, "more than 2^31-2 rows");
    const int32_t NN = (1 << (p->max_depth + 1)) - 1;
    GBT_CHECK(tree->n_nodes >= NN, "tree holds %d nodes, needs %d", tree->n_nodes, NN);
    tree->max_depth = p->max_depth;
    if (stats) memset(stats, 0, sizeof(*stats));
    GBT_TRY(set_device(c));
    return train_tree_naive_impl(c, data, label_d, margin_d, p, tree, stats);
}

gbt_status gbt_train_tree(gbt_ctx *c, const gbt_matrix *data, const float *label_d, float *margin_d,
                          const gbt_train_params *p, gbt_tree *tree, gbt_tree_stats *stats)
{
    GBT_CHECK(c && data && p && tree && tree->nodes, "gbt_train_tree: NULL argument");
    GBT_CHECK(data->n_rows == 0 || (label_d && margin_d), "gbt_train_tree: NULL labels/margins");
    GBT_TRY(hist_check_feature_bins(data));
    GBT_CHECK(p->max_depth >= 0 && p->max_depth <= 20, "max_depth %d outside [0, 20]", p->max_depth);
    GBT_CHECK(p->f > 0.0 && p->f <= 1.0, "f %g outside (0, 1]", p->f);
    GBT_CHECK(p->loss == GBT_LOSS_LOGISTIC || p->loss == GBT_LOSS_SQUARED, "unknown loss %d", p->loss);
    GBT_CHECK(data->n_rows < ((int64_t)1 << 31) - 1, "more than 2^31-2 rows");
    const int32_t NN = (1 << (p->max_depth + 1)) - 1;
    GBT_CHECK(tree->n_nodes >= NN, "tree holds %d nodes, needs %d", tree->n_nodes, NN);
    tree->max_depth = p->max_depth;
    if (stats) memset(stats, 0, sizeof(*stats));
    GBT_TRY(set_device(c));
    return train_tree_impl(c, data, label_d, margin_d, p, tree, stats);
}

gbt_status gbt_train_trees(gbt_ctx *c, const gbt_matrix *data, const float *label_d, float *margin_d,
                           const gbt_train_params *p, int32_t n_trees, gbt_tree *trees, gbt_tree_stats *stats)
{
    GBT_CHECK(c && data && p, "gbt_train_trees: NULL argument");
    GBT_CHECK(n_trees >= 0, "n_trees %d < 0", n_trees);
    if (n_trees == 0) return GBT_OK;
    GBT_CHECK(trees, "gbt_train_trees: NULL trees");
    GBT_CHECK(data->n_rows == 0 || (label_d && margin_d), "gbt_train_trees: NULL labels/margins");
    GBT_TRY(hist_check_feature_bins(data));
    GBT_CHECK(p->max_depth >= 0 && p->max_depth <= 20, "max_depth %d outside [0, 20]", p->max_depth);
    GBT_CHECK(p->f > 0.0 && p->f <= 1.0, "f %g outside (0, 1]", p->f);
    GBT_CHECK(p->loss == GBT_LOSS_LOGISTIC || p->loss == GBT_LOSS_SQUARED, "unknown loss %d", p->loss);
    GBT_CHECK(data->n_rows < ((int64_t)1 << 31) - 1, "more than 2^31-2 rows");
    const int32_t NN = (1 << (p->max_depth + 1)) - 1;
    for (int32_t t = 0; t < n_trees; ++t) {
        GBT_CHECK(trees[t].nodes, "trees[%d].nodes is NULL", t);
        GBT_CHECK(trees[t].n_nodes >= NN, "trees[%d] holds %d nodes, needs %d", t, trees[t].n_nodes, NN);
    }
    if (stats) memset(stats, 0, sizeof(*stats) * (size_t)n_trees);
    GBT_TRY(set_device(c));
    gbt_train_params q = *p;
    // With timing on, each tree is read before the next is queued (the
    // timing marks are per tree).
    if (c->timing) {
        for (int32_t t = 0; t < n_trees; ++t) {
            q.iteration = p->iteration + (uint64_t)t;
            GBT_TRY(train_tree_impl(c, data, label_d, margin_d, &q, &trees[t], stats ? &stats[t] : nullptr));
        }
        return GBT_OK;
    }
    // Every tree is queued without waiting for the one before: its first
    // kernels follow the last tree's margin update on the stream, and its
    // sampling keys' exponent is guessed from that tree's on the device.
    // Each tree writes its result into a slot of a ring (S slots, at most 64
    // MiB; sized by the tree depth alone, so a context allocates it once);
    // the ring's halves are read in turn: before tree t reuses the slots of
    // trees t - S .. t - S + H - 1, those are read after the event recorded
    // behind the last of them.  The rest are read once the stream drains.
    const size_t rb = tree_result_bytes(NN);
    const int32_t S = 2 * (int32_t)std::max<int64_t>(1, std::min<int64_t>(32, ((int64_t)32 << 20) / (int64_t)rb));
    const int32_t H = S / 2;
    void *rh, *rd;
    GBT_TRY(tree_io(c, (size_t)S * rb, &rh, &rd));
    std::vector<TreePending> pend((size_t)S);
    // sampled trees on device pages: each tree's last kernel resets the
    // sampling state for the next
    const bool carry = p->f < 1.0 && !any_host_pages(data);
    int32_t n_read = 0;
    auto read_to = [&](int32_t end) -> gbt_status {
        for (; n_read < end; ++n_read)
            GBT_TRY(train_tree_finish(c, pend[n_read % S], &trees[n_read], stats ? &stats[n_read] : nullptr));
        return GBT_OK;
    };
    for (int32_t t = 0; t < n_trees; ++t) {
        if (t >= S && t % H == 0) {
            GBT_HIP(hipEventSynchronize(pend[(t - S + H - 1) % S].done));
            GBT_TRY(read_to(t - S + H));
        }
        // the event behind the last tree of a half whose slots are reused
        const int32_t g = t / H;
        hipEvent_t ev = nullptr;
        if ((t + 1) % H == 0 && (int64_t)n_trees > (int64_t)(g + 2) * H) GBT_TRY(tree_event(c, g & 1, &ev));
        q.iteration = p->iteration + (uint64_t)t;
        GBT_TRY(train_tree_enqueue(c, data, label_d, margin_d, &q, stats != nullptr, (char *)rh + (size_t)(t % S) * rb,
                                   (char *)rd + (size_t)(t % S) * rb, ev, t > 0, carry && t > 0,
                                   carry && t + 1 < n_trees, &pend[t % S]));
    }
    GBT_HIP(hipStreamSynchronize(c->stream));
    GBT_TRY(read_to(n_trees));
    return GBT_OK;
}

gbt_status gbt_update_leaves(gbt_ctx *c, gbt_tree *tree, const gbt_train_params *tp, const gbt_matrix *data,
                             const int32_t *rows_d, const int32_t *position_d, int64_t n_pos, float *margin_d)
{
    GBT_CHECK(c && tree && tree->nodes && tp && data, "gbt_update_leaves: NULL argument");
    GBT_CHECK(data->n_rows == 0 || margin_d, "margins are NULL");
    GBT_CHECK(n_pos >= 0 && n_pos <= data->n_rows, "n_pos %lld outside [0, %lld]", (long long)n_pos,
              (long long)data->n_rows);
    GBT_CHECK(n_pos == 0 || position_d, "positions are NULL");
    GBT_TRY(set_device(c));
    gbt_node *nodes_d;
    int64_t *offs_d;
    GBT_TRY(upload_trees(c, tree, 1, &nodes_d, &offs_d));
    k_leaf_values<<<blocks(tree->n_nodes), 256, 0, c->stream>>>(nodes_d, tree->n_nodes, tree->exp_g,
                                                               tree->exp_h, tp->lambda, tp->eta);
    GBT_LAUNCHED();
    // rows with known leaves first (marked done), then the traversal of the rest
    uint32_t *done = nullptr;
    unsigned long long *bad = nullptr;
    if (n_pos > 0) {
        const int64_t words = (data->n_rows + 31) / 32;
        GBT_TRY(scratch_t(c, kScrPartFlags, (size_t)words + 2 * sizeof(unsigned long long) / 4, &done));
        const int64_t at = (words + 1) & ~(int64_t)1;  // 8-byte aligned, after the bits
        bad = (unsigned long long *)(done + at);
        k_fill_u32<<<blocks(at + 2), 256, 0, c->stream>>>(done, at + 2, 0u);
        GBT_LAUNCHED();
        k_margin_add_positions<<<blocks(n_pos), 256, 0, c->stream>>>(rows_d, position_d, n_pos, data->n_rows,
                                                                     nodes_d, tree->n_nodes, margin_d, done, bad);
        GBT_LAUNCHED();
    }
    Geo geo = geo_of(data);
    GBT_TRY(for_each_chunk(
        c, data,
        [&](const uint32_t *words, int64_t row0, int64_t rows) -> gbt_status {
            if (geo.row_words <= kWalkMaxWords)
                k_margin_add_tree<true><<<blocks(rows), kWalkThreads, walk_lds_bytes(geo), c->stream>>>(
                    words, rows, geo, nodes_d, tree->n_nodes, margin_d + row0, done, row0);
            else
                k_margin_add_tree<false><<<blocks(rows), kWalkThreads, 0, c->stream>>>(
                    words, rows, geo, nodes_d, tree->n_nodes, margin_d + row0, done, row0);
            GBT_LAUNCHED();
            return GBT_OK;
        },
        nullptr));
    GBT_HIP(hipMemcpyAsync(tree->nodes, nodes_d, tree->n_nodes * sizeof(gbt_node), hipMemcpyDeviceToHost,
                           c->stream));
    unsigned long long n_bad = 0;
    if (bad) GBT_HIP(hipMemcpyAsync(&n_bad, bad, sizeof(n_bad), hipMemcpyDeviceToHost, c->stream));
    GBT_HIP(hipStreamSynchronize(c->stream));
    GBT_CHECK(n_bad == 0,
              "%llu of %lld positions name no leaf of the tree or no new row of the data (those rows were "
              "updated by traversal)",
              n_bad, (long long)n_pos);
    return GBT_OK;
}

gbt_status gbt_predict(gbt_ctx *c, const gbt_tree *trees, int32_t n_trees, const gbt_input *raw,
                       const gbt_matrix *binned, float base_margin, float *margin_out_d)
{
    GBT_CHECK(c && (trees || n_trees == 0) && n_trees >= 0, "gbt_predict: bad trees");
    GBT_CHECK((raw != nullptr) != (binned != nullptr), "give exactly one of raw and binned input");
    GBT_TRY(set_device(c));
    gbt_node *nodes_d = nullptr;
    int64_t *offs_d = nullptr;
    if (n_trees) GBT_TRY(upload_trees(c, trees, n_trees, &nodes_d, &offs_d));
    if (binned) {
        GBT_CHECK(binned->n_rows == 0 || margin_out_d, "output is NULL");
        Geo geo = geo_of(binned);
        GBT_TRY(for_each_chunk(
            c, binned,
            [&](const uint32_t *words, int64_t row0, int64_t rows) -> gbt_status {
                if (geo.row_words <= kWalkMaxWords)
                    k_predict_binned<true><<<blocks(rows), kWalkThreads, walk_lds_bytes(geo), c->stream>>>(
                        words, rows, geo, nodes_d, offs_d, n_trees, base_margin, margin_out_d + row0);
                else
                    k_predict_binned<false><<<blocks(rows), kWalkThreads, 0, c->stream>>>(
                        words, rows, geo, nodes_d, offs_d, n_trees, base_margin, margin_out_d + row0);
                GBT_LAUNCHED();
                return GBT_OK;
            },
            nullptr));
    } else {
        GBT_CHECK(raw->location == GBT_LOC_DEVICE, "raw prediction input must be device resident");
        GBT_CHECK(raw->n_rows >= 0, "n_rows < 0");
        if (raw->n_rows) {
            GBT_CHECK(margin_out_d, "output is NULL");
            if (raw->kind == GBT_INPUT_DENSE_F32) {
                GBT_CHECK(raw->values && raw->ld >= raw->n_cols, "bad dense input");
                k_predict_raw_dense<<<blocks(raw->n_rows), 256, 0, c->stream>>>(
                    raw->values, raw->n_rows, raw->ld, nodes_d, offs_d, n_trees, base_margin, margin_out_d);
            } else {
                GBT_CHECK(raw->indptr && (raw->nnz == 0 || (raw->indices && raw->values)), "bad CSR input");
                k_predict_raw_csr<<<blocks(raw->n_rows), 256, 0, c->stream>>>(
                    raw->indptr, raw->indices, raw->values, raw->n_rows, nodes_d, offs_d, n_trees, base_margin,
                    margin_out_d);
            }
            GBT_LAUNCHED();
        }
    }
    GBT_HIP(hipStreamSynchronize(c->stream));
    return GBT_OK;
}

}  // extern "C"
