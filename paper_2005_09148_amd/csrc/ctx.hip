// ctx.hip -- context, error model and the budgeted device allocator.
#include "common.h"
#include "hist_impl.h"

#include <mutex>

#include <cerrno>
#include <cstring>
#include <unistd.h>

namespace gbt {

static thread_local std::string g_last_error;

gbt_status set_error(gbt_status code, const char *fmt, ...)
{
    char buf[1024];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return code;
}

gbt_status hip_error(hipError_t e, const char *what, const char *file, int line)
{
    gbt_status code = (e == hipErrorOutOfMemory || e == hipErrorMemoryAllocation) ? GBT_E_OOM
                                                                                  : GBT_E_DEVICE;
    return set_error(code, "%s failed: %s (%s:%d)", what, hipGetErrorString(e), file, line);
}

gbt_status set_device(gbt_ctx *c)
{
    GBT_HIP(hipSetDevice(c->device));
    return GBT_OK;
}

gbt_status dev_alloc(gbt_ctx *c, size_t bytes, void **p)
{
    *p = nullptr;
    if (bytes == 0) bytes = 256;
    if (c->budget && c->used + bytes > c->budget)
        return set_error(GBT_E_BUDGET,
                         "device budget exceeded: %llu bytes held + %llu requested > %llu",
                         (unsigned long long)c->used, (unsigned long long)bytes,
                         (unsigned long long)c->budget);
    hipError_t e = hipMalloc(p, bytes);
    if (e != hipSuccess) {
        *p = nullptr;
        (void)hipGetLastError();
        return set_error(GBT_E_OOM, "hipMalloc(%llu) failed: %s", (unsigned long long)bytes,
                         hipGetErrorString(e));
    }
    c->used += bytes;
    if (c->used > c->peak) c->peak = c->used;
    return GBT_OK;
}

void dev_free(gbt_ctx *c, void *p, size_t bytes)
{
    if (!p) return;
    if (bytes == 0) bytes = 256;
    (void)hipFree(p);
    c->used -= bytes;
}

gbt_status host_io(gbt_ctx *c, size_t bytes, void **host, void **dev)
{
    if (c->hio_bytes < bytes) {
        GBT_HIP(hipStreamSynchronize(c->stream));
        if (c->hio) GBT_HIP(hipHostFree(c->hio));
        c->hio = c->hio_d = nullptr;
        c->hio_bytes = 0;
        const size_t sz = std::max<size_t>(bytes, 1 << 16);
        GBT_HIP(hipHostMalloc(&c->hio, sz, hipHostMallocMapped | hipHostMallocCoherent));
        GBT_HIP(hipHostGetDevicePointer(&c->hio_d, c->hio, 0));
        c->hio_bytes = sz;
    }
    *host = c->hio;
    *dev = c->hio_d;
    return GBT_OK;
}

gbt_status tree_io(gbt_ctx *c, size_t bytes, void **host, void **dev)
{
    if (c->tres_bytes < bytes) {
        GBT_HIP(hipStreamSynchronize(c->stream));
        if (c->tres) GBT_HIP(hipHostFree(c->tres));
        c->tres = c->tres_d = nullptr;
        c->tres_bytes = 0;
        const size_t sz = std::max<size_t>(bytes, 1 << 16);
        GBT_HIP(hipHostMalloc(&c->tres, sz, hipHostMallocMapped | hipHostMallocCoherent));
        GBT_HIP(hipHostGetDevicePointer(&c->tres_d, c->tres, 0));
        c->tres_bytes = sz;
    }
    *host = c->tres;
    *dev = c->tres_d;
    return GBT_OK;
}

gbt_status tree_event(gbt_ctx *c, int i, hipEvent_t *ev)
{
    while ((int)c->tres_ev.size() <= i) {
        hipEvent_t e;
        GBT_HIP(hipEventCreateWithFlags(&e, hipEventDisableTiming));
        c->tres_ev.push_back(e);
    }
    *ev = c->tres_ev[i];
    return GBT_OK;
}

size_t scratch_bytes(const gbt_ctx *c, int slot)
{
    return slot < (int)c->scratch.size() ? c->scratch[slot].bytes : 0;
}

gbt_status scratch(gbt_ctx *c, int slot, size_t bytes, void **p)
{
    if ((int)c->scratch.size() <= slot) c->scratch.resize(slot + 1);
    auto &s = c->scratch[slot];
    if (s.bytes < bytes) {
        // the stream may still use the old buffer
        GBT_HIP(hipStreamSynchronize(c->stream));
        dev_free(c, s.p, s.bytes);
        s.p = nullptr;
        s.bytes = 0;
        size_t want = bytes + bytes / 8 + 4096;  // slack so small growth does not reallocate
        GBT_TRY(dev_alloc(c, want, &s.p));
        s.bytes = want;
    }
    *p = s.p;
    return GBT_OK;
}

gbt_status file_read(int fd, void *dst, size_t bytes, int64_t off)
{
    char *p = (char *)dst;
    while (bytes) {
        ssize_t k = pread(fd, p, bytes, (off_t)off);
        if (k < 0 && errno == EINTR) continue;
        if (k <= 0) return set_error(GBT_E_IO, "page file read failed: %s", k < 0 ? strerror(errno) : "end of file");
        p += k;
        off += k;
        bytes -= (size_t)k;
    }
    return GBT_OK;
}

gbt_status file_write(int fd, const void *src, size_t bytes, int64_t off)
{
    const char *p = (const char *)src;
    while (bytes) {
        ssize_t k = pwrite(fd, p, bytes, (off_t)off);
        if (k < 0 && errno == EINTR) continue;
        if (k <= 0) return set_error(GBT_E_IO, "page file write failed: %s", k < 0 ? strerror(errno) : "no progress");
        p += k;
        off += k;
        bytes -= (size_t)k;
    }
    return GBT_OK;
}

bool scratch_fits(const gbt_ctx *c, int slot, size_t bytes)
{
    const size_t have = slot < (int)c->scratch.size() ? c->scratch[slot].bytes : 0;
    if (have >= bytes || !c->budget) return true;
    const size_t want = bytes + bytes / 8 + 4096;
    return c->used - have + want <= c->budget;
}

static int next_event(gbt_ctx *c)
{
    if (c->events_used == (int)c->events.size()) {
        hipEvent_t e;
        if (hipEventCreate(&e) != hipSuccess) return -1;
        c->events.push_back(e);
    }
    return c->events_used++;
}

int timer_begin(gbt_ctx *c, int phase)
{
    if (c->timing == 0 || (c->timing == 1 && phase != kPhHist)) return -1;
    int a = next_event(c), b = next_event(c);
    if (a < 0 || b < 0) return -1;
    (void)hipEventRecord(c->events[a], c->stream);
    c->marks.push_back({a, b, phase});
    return (int)c->marks.size() - 1;
}

int timer_begin_launch(gbt_ctx *c, int phase)
{
    if (c->timing == 0 || (c->timing == 1 && phase != kPhHist)) return -1;
    int a = next_event(c), b = next_event(c);
    if (a < 0 || b < 0) return -1;
    c->marks.push_back({a, b, phase});
    return (int)c->marks.size() - 1;
}

void timer_events(gbt_ctx *c, int mark, hipEvent_t *a, hipEvent_t *b)
{
    *a = c->events[c->marks[mark].a];
    *b = c->events[c->marks[mark].b];
}

void timer_end(gbt_ctx *c, int mark)
{
    if (mark < 0) return;
    (void)hipEventRecord(c->events[c->marks[mark].b], c->stream);
}

void timer_collect(gbt_ctx *c, double *ms)
{
    if (!c->marks.empty()) {
        (void)hipStreamSynchronize(c->stream);
        for (auto &mk : c->marks) {
            float t = 0.f;
            if (hipEventElapsedTime(&t, c->events[mk.a], c->events[mk.b]) == hipSuccess && ms)
                ms[mk.phase] += t;
        }
    }
    c->marks.clear();
    c->events_used = 0;
}

int32_t ceil_log2_u64(uint64_t v)
{
    int32_t b = 0;
    while (b < 64 && ((uint64_t)1 << b) < v) ++b;
    return b;
}

}  // namespace gbt

using namespace gbt;

extern "C" {

int32_t gbt_abi_version(void) { return GBT_ABI_VERSION; }

const char *gbt_last_error(void) { return g_last_error.c_str(); }

gbt_status gbt_ctx_create(int32_t device, uint64_t budget_bytes, void *hip_stream, gbt_ctx **out)
{
    if (!out) return set_error(GBT_E_INVALID, "gbt_ctx_create: out is NULL");
    *out = nullptr;
    int n = 0;
    GBT_HIP(hipGetDeviceCount(&n));
    if (device < 0 || device >= n)
        return set_error(GBT_E_INVALID, "gbt_ctx_create: device %d of %d", device, n);
    GBT_HIP(hipSetDevice(device));
    hipDeviceProp_t prop;
    GBT_HIP(hipGetDeviceProperties(&prop, device));
    if (std::string(prop.gcnArchName).find("gfx950") == std::string::npos)
        return set_error(GBT_E_UNSUPPORTED, "libgbt is built for gfx950; device %d is %s", device,
                         prop.gcnArchName);
    auto *c = new gbt_ctx();
    c->device = device;
    c->budget = budget_bytes;
    c->stream = (hipStream_t)hip_stream;
    hipError_t e = hipStreamCreateWithFlags(&c->side, hipStreamNonBlocking);
    if (e != hipSuccess) {
        delete c;
        return hip_error(e, "hipStreamCreateWithFlags", __FILE__, __LINE__);
    }
    // the device address of gbt_build_hist_noalloc's static scratch on this
    // device (resolved once per device, with the device current)
    const gbt_status ss = static_scratch_init(device);
    if (ss != GBT_OK) {
        (void)hipStreamDestroy(c->side);
        delete c;
        return ss;
    }
    *out = c;
    return GBT_OK;
}

gbt_status gbt_ctx_destroy(gbt_ctx *c)
{
    if (!c) return GBT_OK;
    (void)hipSetDevice(c->device);
    (void)hipStreamSynchronize(c->stream);
    (void)hipStreamSynchronize(c->side);
    for (auto &s : c->scratch) dev_free(c, s.p, s.bytes);
    if (c->hio) (void)hipHostFree(c->hio);
    if (c->tres) (void)hipHostFree(c->tres);
    for (auto e : c->tres_ev) (void)hipEventDestroy(e);
    for (void *p : c->disk_stage)
        if (p) (void)hipHostFree(p);
    for (auto e : c->events) (void)hipEventDestroy(e);
    (void)hipStreamDestroy(c->side);
    delete c;
    return GBT_OK;
}

gbt_status gbt_ctx_memory(gbt_ctx *c, uint64_t *used, uint64_t *peak)
{
    if (!c) return set_error(GBT_E_INVALID, "gbt_ctx_memory: ctx is NULL");
    if (used) *used = c->used;
    if (peak) *peak = c->peak;
    return GBT_OK;
}

gbt_status gbt_ctx_set_timing(gbt_ctx *c, int32_t enable)
{
    if (!c) return set_error(GBT_E_INVALID, "gbt_ctx_set_timing: ctx is NULL");
    c->timing = enable < 0 ? 0 : (enable > 2 ? 2 : enable);
    return GBT_OK;
}

gbt_status gbt_ctx_set_hist_kernel(gbt_ctx *c, int32_t choice)
{
    if (!c) return set_error(GBT_E_INVALID, "gbt_ctx_set_hist_kernel: ctx is NULL");
    if (choice != GBT_HIST_AUTO && choice != GBT_HIST_PLAIN && choice != GBT_HIST_ROTATED)
        return set_error(GBT_E_INVALID, "gbt_ctx_set_hist_kernel: unknown kernel %d", choice);
    c->hist_kernel = choice;
    return GBT_OK;
}

gbt_status gbt_ctx_set_compaction(gbt_ctx *c, int32_t mode)
{
    if (!c) return set_error(GBT_E_INVALID, "gbt_ctx_set_compaction: ctx is NULL");
    if (mode != GBT_COMPACT_AUTO && mode != GBT_COMPACT_STREAM && mode != GBT_COMPACT_GATHER)
        return set_error(GBT_E_INVALID, "gbt_ctx_set_compaction: unknown mode %d", mode);
    c->compaction = mode;
    return GBT_OK;
}

gbt_status gbt_ctx_set_stream_chunk_rows(gbt_ctx *c, int64_t rows)
{
    if (!c) return set_error(GBT_E_INVALID, "gbt_ctx_set_stream_chunk_rows: ctx is NULL");
    if (rows < 0 || rows > ((int64_t)1 << 30))
        return set_error(GBT_E_INVALID, "gbt_ctx_set_stream_chunk_rows: %lld rows outside [0, 2^30]",
                         (long long)rows);
    c->stream_chunk_rows = rows ? rows : ((int64_t)1 << 22);
    return GBT_OK;
}

}  // extern "C"
