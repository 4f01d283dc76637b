// scan.hip -- device-wide exclusive prefix sums (reduce, spine, downsweep).
// Used by the compaction behind sampling and by the stable partition.
#include "common.h"
#include "wave_impl.h"

namespace gbt {

constexpr int kScanThreads = 256;
constexpr int kScanItems = 16;
constexpr int kScanTile = kScanThreads * kScanItems;

// Exclusive scan across a 256-thread block; returns the thread's offset and
// the block total.
__device__ inline int32_t block_exclusive_scan(int32_t v, int32_t *lds4, int32_t *total)
{
    int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    const int32_t x = wave_incl_sum(v);
    if (lane == 63) lds4[wid] = x;
    __syncthreads();
    int32_t off = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < kScanThreads / 64; ++w) {
        int32_t t = lds4[w];
        if (w < wid) off += t;
        tot += t;
    }
    __syncthreads();
    *total = tot;
    return x - v + off;
}

template <typename T>
__global__ void __launch_bounds__(kScanThreads) k_scan_reduce(const T *__restrict__ in, int64_t n,
                                                              int32_t *__restrict__ bsum)
{
    __shared__ int32_t lds4[kScanThreads / 64];
    int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
    int32_t s = 0;
#pragma unroll
    for (int k = 0; k < kScanItems; ++k)
        if (base + k < n) s += (int32_t)in[base + k];
    int32_t tot;
    block_exclusive_scan(s, lds4, &tot);
    if (threadIdx.x == 0) bsum[blockIdx.x] = tot;
}

// One block scans the per-tile sums (in place, exclusive) and writes the total
// (also to total_host, pinned host memory, when given).
__global__ void __launch_bounds__(1024) k_scan_spine(int32_t *__restrict__ bsum, int64_t nb,
                                                     int32_t *__restrict__ total_out,
                                                     int32_t *__restrict__ total_host = nullptr)
{
    __shared__ int32_t lds16[16];
    __shared__ int32_t carry;
    if (threadIdx.x == 0) carry = 0;
    __syncthreads();
    int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    for (int64_t base = 0; base < nb; base += 1024) {
        int64_t i = base + threadIdx.x;
        int32_t v = i < nb ? bsum[i] : 0;
        const int32_t x = wave_incl_sum(v);
        if (lane == 63) lds16[wid] = x;
        __syncthreads();
        int32_t off = carry, tot = 0;
        for (int w = 0; w < 16; ++w) {
            if (w < wid) off += lds16[w];
            tot += lds16[w];
        }
        if (i < nb) bsum[i] = x - v + off;
        __syncthreads();
        if (threadIdx.x == 0) carry += tot;
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        *total_out = carry;
        // the host may poll it while later kernels run
        if (total_host) __hip_atomic_store(total_host, carry, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    }
}

template <typename T>
__global__ void __launch_bounds__(kScanThreads) k_scan_down(const T *__restrict__ in, int64_t n,
                                                            const int32_t *__restrict__ boff,
                                                            int32_t *__restrict__ out)
{
    __shared__ int32_t lds4[kScanThreads / 64];
    int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
    int32_t v[kScanItems];
    int32_t s = 0;
#pragma unroll
    for (int k = 0; k < kScanItems; ++k) {
        v[k] = base + k < n ? (int32_t)in[base + k] : 0;
        s += v[k];
    }
    int32_t tot;
    int32_t run = block_exclusive_scan(s, lds4, &tot) + boff[blockIdx.x];
#pragma unroll
    for (int k = 0; k < kScanItems; ++k) {
        if (base + k < n) out[base + k] = run;
        run += v[k];
    }
}

template <typename T>
static gbt_status scan_impl(gbt_ctx *c, const T *in, int64_t n, int32_t *out)
{
    if (n < 0 || n >= ((int64_t)1 << 31) - 1)
        return set_error(GBT_E_UNSUPPORTED, "scan of %lld items (limit 2^31-2)", (long long)n);
    int64_t nb = (n + kScanTile - 1) / kScanTile;
    if (nb == 0) {
        GBT_HIP(hipMemsetAsync(out, 0, sizeof(int32_t), c->stream));
        return GBT_OK;
    }
    int32_t *bsum;
    GBT_TRY(scratch_t(c, kScrScan, (size_t)nb, &bsum));
    k_scan_reduce<T><<<(unsigned)nb, kScanThreads, 0, c->stream>>>(in, n, bsum);
    GBT_LAUNCHED();
    k_scan_spine<<<1, 1024, 0, c->stream>>>(bsum, nb, out + n);
    GBT_LAUNCHED();
    k_scan_down<T><<<(unsigned)nb, kScanThreads, 0, c->stream>>>(in, n, bsum, out);
    GBT_LAUNCHED();
    return GBT_OK;
}

gbt_status scan_tiles_u8(gbt_ctx *c, const uint8_t *in, int64_t n, int32_t *tile_off)
{
    if (n < 0 || n >= ((int64_t)1 << 31) - 1)
        return set_error(GBT_E_UNSUPPORTED, "scan of %lld items (limit 2^31-2)", (long long)n);
    int64_t nb = (n + kScanTile - 1) / kScanTile;
    if (nb > 0) {
        k_scan_reduce<uint8_t><<<(unsigned)nb, kScanThreads, 0, c->stream>>>(in, n, tile_off);
        GBT_LAUNCHED();
    }
    k_scan_spine<<<1, 1024, 0, c->stream>>>(tile_off, nb, tile_off + nb);
    GBT_LAUNCHED();
    return GBT_OK;
}

gbt_status scan_tile_counts(gbt_ctx *c, int32_t *tile_cnt, int64_t tiles, int32_t *total_host)
{
    k_scan_spine<<<1, 1024, 0, c->stream>>>(tile_cnt, tiles, tile_cnt + tiles, total_host);
    GBT_LAUNCHED();
    return GBT_OK;
}

gbt_status scan_u8(gbt_ctx *c, const uint8_t *in, int64_t n, int32_t *out)
{
    return scan_impl<uint8_t>(c, in, n, out);
}

gbt_status scan_u32(gbt_ctx *c, const uint32_t *in, int64_t n, int32_t *out)
{
    return scan_impl<uint32_t>(c, in, n, out);
}

}  // namespace gbt
