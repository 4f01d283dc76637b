// common.h -- internals shared by the libgbt translation units: context,
// budgeted device allocator, error model, matrix/page objects and the
// device-side ELLPACK decoding helpers.
#pragma once

#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <string>
#include <vector>

#include "gbt.h"

namespace gbt {

// ---------------------------------------------------------------- errors
gbt_status set_error(gbt_status code, const char *fmt, ...);
gbt_status hip_error(hipError_t e, const char *what, const char *file, int line);

#define GBT_HIP(call)                                                                  \
    do {                                                                               \
        hipError_t e_ = (call);                                                        \
        if (e_ != hipSuccess) return ::gbt::hip_error(e_, #call, __FILE__, __LINE__); \
    } while (0)

#define GBT_TRY(expr)                    \
    do {                                 \
        gbt_status s_ = (expr);          \
        if (s_ != GBT_OK) return s_;     \
    } while (0)

#define GBT_CHECK(cond, ...)                                              \
    do {                                                                  \
        if (!(cond)) return ::gbt::set_error(GBT_E_INVALID, __VA_ARGS__); \
    } while (0)

// Kernel launches: check the launch itself (configuration errors).
#define GBT_LAUNCHED() GBT_HIP(hipGetLastError())

constexpr int kXcds = 8;         // gfx950: 8 XCDs of 32 CUs
// Spread copies of the histogram update counter, one 128-byte line apart
// (copy k at word k * kUpdStride), so that the workgroups' atomics do not
// serialize on one line.
constexpr int kUpdCounters = 32;
constexpr int kUpdStride = 16;
constexpr int kUpdWords = kUpdCounters * kUpdStride;
constexpr int kCUs = 256;

// Map a linear workgroup id so that logically adjacent ids run on the same
// XCD (the hardware deals workgroups round-robin over the XCDs).
__device__ inline uint32_t xcd_remap(uint32_t b, uint32_t n)
{
    uint32_t xcd = b % kXcds, local = b / kXcds;
    uint32_t per = n / kXcds, rem = n % kXcds;
    return xcd < rem ? xcd * (per + 1) + local : rem * (per + 1) + (xcd - rem) * per + local;
}

}  // namespace gbt

// ---------------------------------------------------------------- context
struct gbt_ctx {
    int device = 0;
    hipStream_t stream = nullptr;   // compute stream (caller's)
    hipStream_t side = nullptr;     // host-to-device page copies
    uint64_t budget = 0;            // 0 = unlimited
    uint64_t used = 0, peak = 0;
    int timing = 0;  // 0 off, 1 histogram kernel only, 2 every phase
    int hist_kernel = GBT_HIST_AUTO;
    int compaction = GBT_COMPACT_AUTO;
    int64_t stream_chunk_rows = (int64_t)1 << 22;  // rows per streamed chunk of a host or disk page
    struct Mark {
        int a, b;    // indices into events
        int phase;
    };
    std::vector<hipEvent_t> events;  // pool, reused
    int events_used = 0;
    std::vector<Mark> marks;
    struct Scratch {
        void *p = nullptr;
        size_t bytes = 0;
    };
    std::vector<Scratch> scratch;   // reusable workspaces, by slot id
    // pinned host memory the kernels write results into (read after a sync)
    void *hio = nullptr;
    void *hio_d = nullptr;
    size_t hio_bytes = 0;
    // pinned memory a tree's last kernels write the tree into (one slot per
    // tree of a run of trees whose results are read together), and events
    // recorded after trees whose slot is reused within a run
    void *tres = nullptr;
    void *tres_d = nullptr;
    size_t tres_bytes = 0;
    std::vector<hipEvent_t> tres_ev;
    // what the column-copy workspace holds: a matrix's own device page
    // (kept across trees, since such a page does not change)
    uint64_t cols_uid = 0;
    const void *cols_page = nullptr;
    const void *cols_at = nullptr;
    int64_t cols_rows = 0;
    // pinned buffers that disk pages are read into before their copy
    void *disk_stage[2] = {nullptr, nullptr};
    size_t disk_stage_bytes = 0;
    // the MVS key exponent of the last tree with sampling, for its row
    // count and lambda (the next tree's gradient pass guesses it)
    int32_t key_e_last = 0;
    int64_t key_n_last = -1;
    double key_lambda_last = 0.0;
    // whether the last MVS threshold needed the radix descent (the next
    // tree then compacts only after the threshold is complete)
    bool mvs_descent_last = false;
};

namespace gbt {

// Phase timing: events recorded on the context stream around kernel
// groups, read once after the stream has drained.
enum Phase { kPhSample = 0, kPhHist, kPhHistAux, kPhSplit, kPhMargin, kPhCount };
int timer_begin(gbt_ctx *c, int phase);   // -1 when timing is off
void timer_end(gbt_ctx *c, int mark);
// A mark whose two events one kernel launch fills itself (its start and end
// timestamps, hipExtLaunchKernel): no timer_end.
int timer_begin_launch(gbt_ctx *c, int phase);
void timer_events(gbt_ctx *c, int mark, hipEvent_t *a, hipEvent_t *b);
void timer_collect(gbt_ctx *c, double *ms_per_phase);  // adds, then resets

gbt_status dev_alloc(gbt_ctx *c, size_t bytes, void **p);
void dev_free(gbt_ctx *c, void *p, size_t bytes);
// Grow-only workspace in slot `slot` of the context.
gbt_status scratch(gbt_ctx *c, int slot, size_t bytes, void **p);
// Whether scratch(c, slot, bytes) stays within the context's byte budget
// (for optional workspaces that are skipped when it would not).
// Whole reads and writes of page files at a byte offset (retried on short
// transfers and EINTR).
gbt_status file_read(int fd, void *dst, size_t bytes, int64_t off);
gbt_status file_write(int fd, const void *src, size_t bytes, int64_t off);
bool scratch_fits(const gbt_ctx *c, int slot, size_t bytes);
// The bytes workspace `slot` holds now (0 before its first use).
size_t scratch_bytes(const gbt_ctx *c, int slot);
// Grow-only pinned host buffer that kernels write into: *host for the host,
// *dev for kernels.  The stream must not be using it (the call syncs
// before growing).
gbt_status host_io(gbt_ctx *c, size_t bytes, void **host, void **dev);
// The tree driver's pinned result memory, grown like host_io's.
gbt_status tree_io(gbt_ctx *c, size_t bytes, void **host, void **dev);
// Event i of the tree driver (created on first use).
gbt_status tree_event(gbt_ctx *c, int i, hipEvent_t *ev);
gbt_status set_device(gbt_ctx *c);

enum ScratchSlot {
    kScrGpair = 0,   // float (g, h) of all rows
    kScrKeys,        // MVS keys
    kScrFlags,       // keep flags
    kScrPos,         // scan of the keep flags
    kScrMisc,        // threshold radix histogram
    kScrState,       // SampleState
    kScrSampled,     // the sampled page
    kScrSel,         // global ids of the sampled rows
    kScrGw,          // reweighted (g', h') in double
    kScrQ,           // fixed-point (q_g, q_h)
    kScrRows, kScrRowsTmp, kScrPosition, kScrSlotA, kScrSlotB, kScrCand,
    kScrHistA, kScrHistB,
    kScrNodes,       // DevNode table
    kScrEvalNodes,   // EvalNode list
    kScrSplits,      // gbt_split per evaluated node
    kScrEval,        // per feature-block candidates
    kScrPartFlags, kScrPartPos,
    kScrWork,        // histogram plan
    kScrUpd,         // histogram update counter
    kScrScan,        // scan block sums
    kScrStage0, kScrStage1,  // streamed page chunks
    kScrLeaf,        // leaf values
    kScrTrees,       // trees for prediction
    kScrSlotNode,    // slot -> node map
    kScrPartials,    // per-chunk partial histograms
    kScrCompact,     // compact tree for the row walk
    kScrPlan,        // device-side level plans (lists, work items, counts)
    kScrPartialsDev, // partial histograms of the device-planned levels
    kScrSlotTbl,     // slot table of a sparse training page
    kScrCols,        // column copy of a dense training page
    kScrCount
};

template <typename T>
gbt_status scratch_t(gbt_ctx *c, int slot, size_t n, T **p)
{
    return scratch(c, slot, n * sizeof(T), reinterpret_cast<void **>(p));
}

}  // namespace gbt

// ---------------------------------------------------------------- matrix
struct GbtPage {
    int64_t row0 = 0;
    int64_t rows = 0;
    uint32_t *words = nullptr;  // device or pinned host (NULL on disk)
    bool host = false;          // pinned host memory
    int fd = -1;                // the page's (unlinked) file, when on disk
    bool streamed() const { return host || fd >= 0; }
};

// A process-unique id per matrix (never reused, unlike an address).
inline uint64_t next_matrix_uid()
{
    static std::atomic<uint64_t> n{0};
    return ++n;
}

struct gbt_matrix {
    gbt_ctx *ctx = nullptr;
    uint64_t uid = next_matrix_uid();
    int64_t n_rows = 0;
    int32_t m = 0;
    int32_t sparse = 0;
    int32_t has_missing = 0;
    int32_t w = 1;
    int32_t stride = 0;
    int32_t row_words = 4;
    uint32_t null_sym = 0;
    int64_t total_bins = 0;
    int64_t page_rows = 0;
    int32_t page_home = GBT_HOME_DEVICE;
    std::vector<int32_t> cut_ptr_h;     // m+1
    std::vector<float> cut_values_h;
    int32_t *cut_ptr_d = nullptr;       // m+1
    float *cut_values_d = nullptr;
    int32_t *bin_ptr_d = nullptr;       // m+1 global bin offsets (cut_ptr[j] + j)
    std::vector<int32_t> bin_ptr_h;
    std::vector<int64_t> feat_count_h;  // sparse: present values per feature in the sketch rows (m)
    std::vector<GbtPage> pages;
    // the histogram kernel's feature groups on the device, cached per kernel kind
    mutable void *groups_d = nullptr;
    mutable size_t groups_bytes = 0;
    mutable int32_t groups_kind = -1;
};

namespace gbt {

// Everything a kernel needs to decode an ELLPACK row.
struct Geo {
    int32_t m;
    int32_t w;
    int32_t stride;
    int32_t row_words;
    uint32_t null_sym;
    uint32_t mask;
    int32_t sparse;
    int32_t pad0;
    int64_t total_bins;
    const int32_t *bin_ptr;  // m+1
};

// null_sym is a value no symbol can take when the matrix has no missing
// value (a dense page without missing values uses every w-bit code).
inline Geo geo_of(const gbt_matrix *mx)
{
    Geo g;
    g.m = mx->m;
    g.w = mx->w;
    g.stride = mx->stride;
    g.row_words = mx->row_words;
    g.null_sym = (mx->sparse || mx->has_missing) ? mx->null_sym : 0xffffffffu;
    g.mask = mx->w >= 32 ? 0xffffffffu : ((1u << mx->w) - 1u);
    g.sparse = mx->sparse;
    g.pad0 = 0;
    g.total_bins = mx->total_bins;
    g.bin_ptr = mx->bin_ptr_d;
    return g;
}

// Symbol in slot s of an ELLPACK row (LSB-first bit stream).  Reads the next
// word only when the symbol straddles a word boundary.
__device__ inline uint32_t row_symbol(const uint32_t *__restrict__ row, int32_t s, int32_t w,
                                      uint32_t mask)
{
    uint32_t bit = (uint32_t)s * (uint32_t)w;
    uint32_t k = bit >> 5, sh = bit & 31u;
    uint32_t v = row[k] >> sh;
    if (sh + (uint32_t)w > 32u) v |= row[k + 1] << (32u - sh);
    return v & mask;
}

// Local bin of feature j in a row, or -1 when missing.
__device__ inline int32_t row_feature_bin(const uint32_t *__restrict__ row, const Geo &g, int32_t j)
{
    if (!g.sparse) {
        uint32_t s = row_symbol(row, j, g.w, g.mask);
        return s == g.null_sym ? -1 : (int32_t)s;
    }
    // the row's symbols are ascending global bins, padded with the null
    // symbol (the largest): binary search for the first symbol >= lo
    const uint32_t lo = (uint32_t)g.bin_ptr[j], hi = (uint32_t)g.bin_ptr[j + 1];
    int32_t a = 0, b = g.stride;
    while (a < b) {
        const int32_t mid = (a + b) >> 1;
        if (row_symbol(row, mid, g.w, g.mask) < lo)
            a = mid + 1;
        else
            b = mid;
    }
    if (a == g.stride) return -1;
    const uint32_t v = row_symbol(row, a, g.w, g.mask);
    return v < hi ? (int32_t)(v - lo) : -1;
}

// Sparse pages: for each row and histogram feature group g, the row's slots
// that hold the group's symbols (the symbols ascend and the groups are
// contiguous bin ranges).  Built by the tree driver for the page it trains
// on, in two layouts: by row (row[r * row_stride + g] = first slot of group
// g, g <= groups), which the histogram passes read (the groups' workgroups
// of one row share its line), and by group (col[g * rows + r] = first |
// (end << 8)), which the partition reads for the split feature's group (a
// node's rows are monotone, so a column line serves several of them).
struct SlotTable {
    const uint8_t *row;       // rows x row_stride; NULL: no table
    const uint16_t *col;      // groups x rows
    const uint8_t *feat_grp;  // m: the group of each feature
    int64_t rows;
    int32_t row_stride;
    int32_t pad0;
};

// row_feature_bin for a sparse row whose feature-j group occupies slots
// [a, e) of the row.
__device__ inline int32_t row_feature_bin_range(const uint32_t *__restrict__ row, const Geo &g, int32_t j,
                                                int32_t a, int32_t e)
{
    const uint32_t lo = (uint32_t)g.bin_ptr[j], hi = (uint32_t)g.bin_ptr[j + 1];
    int32_t b = e;
    while (a < b) {
        const int32_t mid = (a + b) >> 1;
        if (row_symbol(row, mid, g.w, g.mask) < lo)
            a = mid + 1;
        else
            b = mid;
    }
    if (a == e) return -1;
    const uint32_t v = row_symbol(row, a, g.w, g.mask);
    return v < hi ? (int32_t)(v - lo) : -1;
}

// Device node table entry used by the tree driver (heap order).  The split
// record {split, feature, split_bin, default_left} is 16-byte aligned so
// that the partition reads it with one load.
struct __align__(16) DevNode {
    int64_t sum_g, sum_h;
    int64_t begin, end;
    int32_t split;          // 1 if the node splits
    int32_t feature, split_bin;
    int32_t default_left;
    int32_t present;
    int32_t left_child;     // node ids of the children (heap: 2i+1, 2i+2)
    int32_t right_child;
    int32_t slot;           // tree driver: the node's index in its level's list (its histogram slot)
    int64_t pleft;          // partition: left flags before begin (all slots)
    int64_t nleft;          // partition: rows of the segment that go left
    double gain;
    int64_t left_g, left_h, right_g, right_h;
    // tree driver's partition: the tiles of the first and last slot and the
    // left flags of those tiles before the first slot and up to the last
    int32_t tile_b, left_b, tile_e, left_e;
};
static_assert(sizeof(DevNode) % 16 == 0, "DevNode is read with 16-byte loads");

// ---------------------------------------------------------------- scans
// Exclusive prefix sum of n flags (bytes 0/1) or counts (uint32): out[i] for
// i in [0, n], out[n] = total.  Device-wide, deterministic.
gbt_status scan_u8(gbt_ctx *c, const uint8_t *in, int64_t n, int32_t *out);
gbt_status scan_u32(gbt_ctx *c, const uint32_t *in, int64_t n, int32_t *out);
// Exclusive sums of the per-tile counts of n flags (tiles of 4096);
// tile_off[ceil(n/4096)] = total.
gbt_status scan_tiles_u8(gbt_ctx *c, const uint8_t *in, int64_t n, int32_t *tile_off);
// Exclusive sums of `tiles` per-tile counts, in place; tile_cnt[tiles]
// receives the total, and so does *total_host (pinned, device-mapped) when
// given.
gbt_status scan_tile_counts(gbt_ctx *c, int32_t *tile_cnt, int64_t tiles, int32_t *total_host = nullptr);

// ---------------------------------------------------------------- shared launches
gbt_status launch_gradients(gbt_ctx *c, int32_t loss, const float *margin, const float *label,
                            const float *weight, int64_t n, float *gpair);
struct HistWorkspace;
// ws: device memory for the partial histograms and the plan (NULL: the
// context's workspaces)
gbt_status build_hist_impl(gbt_ctx *c, const gbt_matrix *layout, const uint32_t *page,
                           const int64_t *q, const int32_t *rows, const gbt_seg *build,
                           int32_t n_build, const gbt_sub *sub, int32_t n_sub,
                           const int64_t *parent_hist, int64_t *hist, gbt_tree_stats *stats,
                           const HistWorkspace *ws = nullptr);

// Row-major ELLPACK page geometry helpers (host).
int32_t ceil_log2_u64(uint64_t v);

}  // namespace gbt
