// sample.hip -- Eq. 4-5 gradients, Eq. 9 minimal variance sampling with the
// compaction of Alg. 7 (Sec. 3.4), and the exact fixed-point conversion of
// the reweighted gradient pairs.
//
// The sampling threshold T* (least integer T >= 1 with
// sum_{a_i<T} a_i <= (K - #{a_i >= T}) T) is found without sorting: at the
// boundaries of key buckets both #{a >= T} and sum_{a < T} a follow from a
// (count, sum) histogram, so a radix descent over 11-bit digits pins T*
// exactly in ceil(bits/11) passes over the keys.  When T* exceeds every key
// it has the closed form ceil(sum a / K).
#include "sample_impl.h"
#include "wave_impl.h"

#include <chrono>

namespace gbt {

// ------------------------------------------------------------ exp (device)
// Cody & Waite reduction of x by ln 2 (head with 32 significant bits, tail
// the remainder), Taylor polynomial of e^r through r^13 by Horner with fused
// multiply-adds, scaling by 2^k.  Inputs beyond +-708 clamp to +inf / 0.
__device__ inline double cw_exp(double x)
{
    constexpr double kLn2Head = 0x1.62e42fee00000p-1;
    constexpr double kLn2Tail = 0x1.a39ef35793c76p-33;
    constexpr double kInvLn2 = 0x1.71547652b82fep+0;
    // 1/13!, 1/12!, ..., 1/2!, 1/1!, 1/0!
    constexpr double kTaylor[14] = {0x1.6124613a86d09p-33, 0x1.1eed8eff8d898p-29, 0x1.ae64567f544e4p-26,
                                    0x1.27e4fb7789f5cp-22, 0x1.71de3a556c734p-19, 0x1.a01a01a01a01ap-16,
                                    0x1.a01a01a01a01ap-13, 0x1.6c16c16c16c17p-10, 0x1.1111111111111p-7,
                                    0x1.5555555555555p-5,  0x1.5555555555555p-3,  0.5,
                                    1.0,                   1.0};
    if (x != x) return x;
    if (x > 708.0) return __builtin_huge_val();
    if (x < -708.0) return 0.0;
    double k = rint(x * kInvLn2);
    double r = (x - k * kLn2Head) - k * kLn2Tail;
    double p = kTaylor[0];
#pragma unroll
    for (int i = 1; i < 14; ++i) p = fma(p, r, kTaylor[i]);
    return ldexp(p, (int)k);
}

__device__ inline void gradient_pair(int32_t loss, float margin, float label, double *g, double *h)
{
    double z = (double)margin, y = (double)label;
    if (loss == GBT_LOSS_LOGISTIC) {
        double s = 1.0 / (1.0 + cw_exp(-z));
        *g = s - y;
        double hh = s * (1.0 - s);
        *h = hh < 1e-16 ? 1e-16 : hh;
    } else {
        *g = z - y;
        *h = 1.0;
    }
}

__global__ void k_gradients(int32_t loss, const float *__restrict__ margin,
                            const float *__restrict__ label, const float *__restrict__ weight,
                            int64_t n, float2 *__restrict__ gpair)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    double g, h;
    gradient_pair(loss, margin[i], label[i], &g, &h);
    if (weight) {
        double w = (double)weight[i];
        g = g * w;
        h = h * w;
    }
    gpair[i] = make_float2((float)g, (float)h);
}

// Gradients of all rows and the maximum of r over them, as the keys define it
// (from the float-rounded pair).
__global__ void __launch_bounds__(256) k_gradients_rmax(int32_t loss, const float *__restrict__ margin,
                                                        const float *__restrict__ label, int64_t n,
                                                        float2 *__restrict__ gpair, double lambda,
                                                        SampleState *__restrict__ st);

gbt_status launch_gradients(gbt_ctx *c, int32_t loss, const float *margin, const float *label,
                            const float *weight, int64_t n, float *gpair)
{
    if (n == 0) return GBT_OK;
    k_gradients<<<(unsigned)((n + 255) / 256), 256, 0, c->stream>>>(loss, margin, label, weight, n,
                                                                    (float2 *)gpair);
    GBT_LAUNCHED();
    return GBT_OK;
}

// ------------------------------------------------------------ Philox4x64-10
// Salmon et al., SC'11: ten rounds of two 64x64->128 multiplies, the key
// advanced by the Weyl increments between rounds.
// The full 128-bit product of x and a constant m, from four 32 x 32 -> 64
// multiply-adds (no partial sum overflows 64 bits).
__device__ inline void mul_128(uint64_t m, uint64_t x, uint64_t *hi, uint64_t *lo)
{
    const uint64_t ml = (uint32_t)m, mh = m >> 32, xl = (uint32_t)x, xh = x >> 32;
    const uint64_t p0 = xl * ml;
    const uint64_t p1 = xl * mh + (p0 >> 32);
    const uint64_t p2 = xh * ml + (uint32_t)p1;
    *hi = xh * mh + (p1 >> 32) + (p2 >> 32);
    *lo = (p2 << 32) | (uint32_t)p0;
}

// The block of counter (c0, c1, 0, 0) and key (k0, 0): its four words.
__device__ inline void philox_block(uint64_t c0, uint64_t c1, uint64_t k0, uint64_t out[4])
{
    constexpr uint64_t kMul0 = 0xD2E7470EE14C6C93ull, kMul1 = 0xCA5A826395121157ull;
    constexpr uint64_t kWeyl0 = 0x9E3779B97F4A7C15ull, kWeyl1 = 0xBB67AE8584CAA73Bull;
    uint64_t c2 = 0, c3 = 0, k1 = 0;
#pragma unroll
    for (int round = 0; round < 10; ++round) {
        uint64_t p0hi, p0lo, p1hi, p1lo;
        mul_128(kMul0, c0, &p0hi, &p0lo);
        mul_128(kMul1, c2, &p1hi, &p1lo);
        uint64_t n0 = p1hi ^ c1 ^ k0, n2 = p0hi ^ c3 ^ k1;
        c0 = n0;
        c1 = p1lo;
        c2 = n2;
        c3 = p0lo;
        k0 += kWeyl0;
        k1 += kWeyl1;
    }
    out[0] = c0;
    out[1] = c1;
    out[2] = c2;
    out[3] = c3;
}

// ------------------------------------------------------------ block reductions
// 256-thread blocks: wavefront butterfly, then the four wave results in LDS.
__device__ inline unsigned long long block_max_u64(unsigned long long v, unsigned long long *lds4)
{
    v = wave_max(v);
    __syncthreads();
    if ((threadIdx.x & 63) == 0) lds4[threadIdx.x >> 6] = v;
    __syncthreads();
    unsigned long long r = lds4[0];
    for (int w = 1; w < 4; ++w) r = lds4[w] > r ? lds4[w] : r;
    return r;
}

__device__ inline unsigned long long block_sum_u64(unsigned long long v, unsigned long long *lds4)
{
    v = wave_total(v);
    __syncthreads();
    if ((threadIdx.x & 63) == 0) lds4[threadIdx.x >> 6] = v;
    __syncthreads();
    return lds4[0] + lds4[1] + lds4[2] + lds4[3];
}

constexpr int kReduceGrid = 2048;  // blocks of the grid-stride reductions

// ------------------------------------------------------------ MVS keys
template <int kSrc>
__device__ inline void row_gh(const SampleSrc &src, int64_t i, double *g, double *h)
{
    if (kSrc == kSrcGpair) {
        float2 p = src.gpair[i];
        *g = (double)p.x;
        *h = (double)p.y;
    } else {
        // gradients recomputed from margins, rounded to float as if stored
        double gg, hh;
        gradient_pair(src.loss, src.margin[i], src.label[i], &gg, &hh);
        *g = (double)(float)gg;
        *h = (double)(float)hh;
    }
}

// r^2 as r is formed: the square root of this value, rounded, is r.  The
// square root is monotone, so the largest r is the root of the largest r^2
// and the maximum passes need no root per row.
__device__ inline double mvs_r2(double g, double h, double lambda)
{
    return g * g + lambda * (h * h);
}

__device__ inline double mvs_r(double g, double h, double lambda)
{
    return sqrt(mvs_r2(g, h, lambda));
}

// A spread maximum folded by the block's first wave and shared through LDS;
// every thread of the block calls it.
__device__ inline unsigned long long block_fold_max(const Spread &a, unsigned long long *lds1)
{
    if (threadIdx.x < 64) {
        const unsigned long long v = wave_max(threadIdx.x < kSpread ? a[threadIdx.x][0] : 0ull);
        if (threadIdx.x == 0) *lds1 = v;
    }
    __syncthreads();
    return *lds1;
}

template <int kSrc>
__global__ void __launch_bounds__(256) k_mvs_rmax(SampleSrc src, int64_t n, double lambda,
                                                  SampleState *__restrict__ st)
{
    __shared__ unsigned long long lds4[4];
    unsigned long long b = 0;
    bool bad = false;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        double g, h;
        row_gh<kSrc>(src, i, &g, &h);
        const double x = mvs_r2(g, h, lambda);
        bad |= !(x <= 1.7976931348623157e308);  // NaN or infinite
        const unsigned long long xb = __double_as_longlong(x);  // x >= 0: bit order = value order
        b = xb > b ? xb : b;
    }
    if (bad) atomicOr(&st->bad, 1u);
    b = block_max_u64(b, lds4);
    if (threadIdx.x == 0 && b) atomicMax(spread_at(st->rmax, blockIdx.x), b);
}

// a_i = rint(r_i * 2^e), e = 62 - E - L with max r < 2^E; also max and sum
// of the keys and, fused, nothing else.
template <int kSrc>
__global__ void __launch_bounds__(256) k_mvs_keys(SampleSrc src, int64_t n, double lambda,
                                                  int32_t log2n, SampleState *__restrict__ st,
                                                  int64_t *__restrict__ keys)
{
    __shared__ unsigned long long lds4[4], m1;
    int E;
    frexp(sqrt(__longlong_as_double(block_fold_max(st->rmax, &m1))), &E);
    const int32_t e = 62 - E - log2n;
    unsigned long long mx = 0, sm = 0;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        double g, h;
        row_gh<kSrc>(src, i, &g, &h);
        unsigned long long a = (unsigned long long)(long long)rint(ldexp(mvs_r(g, h, lambda), e));
        if (keys) keys[i] = (int64_t)a;
        mx = a > mx ? a : mx;
        sm += a;
    }
    mx = block_max_u64(mx, lds4);
    sm = block_sum_u64(sm, lds4);
    if (threadIdx.x == 0) {
        if (mx) atomicMax(spread_at(st->amax, blockIdx.x), mx);
        if (sm) atomicAdd(spread_at(st->asum, blockIdx.x), sm);
        if (blockIdx.x == 0) st->e_key = e;
    }
}

// Closed form when T* exceeds every key; otherwise the radix descent
// starts on [0, 2^S) with 2^S > amax + 1.  done_host (pinned host memory,
// may be NULL) receives 1 for the closed form, else 0.  check_log2n >= 0:
// the key sums were formed with the exponent in st->e_key, which is first
// checked against the one max r gives (e = 62 - E - check_log2n); when they
// differ nothing else is done and done_host receives 2.  The flag is a
// relaxed store: the host reads nothing else this kernel writes (the
// kernels it queues after reading the flag see the rest in stream order).
__device__ inline void thresh_first(SampleState *__restrict__ st, int64_t K, int32_t *__restrict__ done_host,
                                    int32_t count_mode, int32_t check_log2n)
{
    if (check_log2n >= 0) {
        int E;
        frexp(sqrt(__longlong_as_double(fold_max(st->rmax))), &E);
        if (62 - E - check_log2n != st->e_key) {
            if (done_host) __hip_atomic_store(done_host, 2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
            return;
        }
    }
    unsigned long long amax = fold_max(st->amax), asum = fold_sum(st->asum);
    st->C_above = 0;
    st->F_below = 0;
    st->lo = 0;
    // count mode: no top rows when A = 0; otherwise always a descent
    const bool closed = count_mode ? K <= 0 : (asum + (unsigned long long)K - 1) / (unsigned long long)K > amax + 1;
    if (closed) {
        st->T = count_mode ? 0x7fffffffffffffffll
                           : (long long)((asum + (unsigned long long)K - 1) / (unsigned long long)K);
        st->done = 1;
        st->levels = 0;
        if (done_host) __hip_atomic_store(done_host, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        return;
    }
    if (done_host) __hip_atomic_store(done_host, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    int S = 64 - __clzll((long long)(amax + 1));  // 2^S > amax + 1
    int levels = (S + kDigitBits - 1) / kDigitBits;
    st->shift = (levels - 1) * kDigitBits;
    st->nbuckets = (int32_t)(((1ull << S) + (1ull << st->shift) - 1) >> st->shift);
    st->levels = levels;
    st->done = 0;
    st->T = 0;
}

__global__ void k_mvs_thresh_init(SampleState *__restrict__ st, int64_t K, int32_t *__restrict__ done_host,
                                  int32_t count_mode, int32_t check_log2n)
{
    if (threadIdx.x == 0) thresh_first(st, K, done_host, count_mode, check_log2n);
}

// The T that thresh_first (count_mode 0) leaves in a state whose T was 0:
// the closed form's when the exponent checks and the form holds, else 0.
// Called by a whole wave: lane l folds entry l of the spread sums.
__device__ inline unsigned long long thresh_first_T_wave(const SampleState *__restrict__ st, int64_t K,
                                                         int32_t check_log2n)
{
    static_assert(kSpread <= 64, "one spread entry per lane");
    const int lane = threadIdx.x & 63;
    unsigned long long rm = 0, am = 0, as = 0;
    if (lane < kSpread) {
        rm = st->rmax[lane][0];
        am = st->amax[lane][0];
        as = st->asum[lane][0];
    }
    rm = wave_max(rm);  // r^2 >= 0: the double bits order as integers
    am = wave_max(am);
    as = wave_total(as);
    if (check_log2n >= 0) {
        int E;
        frexp(sqrt(__longlong_as_double(rm)), &E);
        if (62 - E - check_log2n != st->e_key) return 0;
    }
    const unsigned long long Tc = (as + (unsigned long long)K - 1) / (unsigned long long)K;
    return Tc > am + 1 ? Tc : 0;
}

template <int kSrc>
__global__ void __launch_bounds__(256) k_mvs_radix_hist(SampleSrc src, const int64_t *__restrict__ keys,
                                                        int64_t n, double lambda, int32_t log2n,
                                                        const SampleState *__restrict__ st,
                                                        unsigned long long *__restrict__ hcnt,
                                                        unsigned long long *__restrict__ hsum)
{
    __shared__ unsigned int scnt[kDigitBuckets];
    __shared__ unsigned long long ssum[kDigitBuckets];
    if (st->done) return;
    const unsigned long long lo = (unsigned long long)st->lo;
    const int shift = st->shift;
    const int32_t nb = st->nbuckets;
    for (int t = threadIdx.x; t < nb; t += blockDim.x) {
        scnt[t] = 0;
        ssum[t] = 0;
    }
    __syncthreads();
    int32_t e = st->e_key;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        unsigned long long a;
        if (keys) {
            a = (unsigned long long)keys[i];
        } else {
            double g, h;
            row_gh<kSrc>(src, i, &g, &h);
            a = (unsigned long long)(long long)rint(ldexp(mvs_r(g, h, lambda), e));
        }
        if (a < lo) continue;
        unsigned long long b = (a - lo) >> shift;
        if (b >= (unsigned long long)nb) continue;
        atomicAdd(&scnt[b], 1u);
        atomicAdd(&ssum[b], a);
    }
    __syncthreads();
    for (int t = threadIdx.x; t < nb; t += blockDim.x) {
        if (scnt[t]) {
            atomicAdd(&hcnt[t], (unsigned long long)scnt[t]);
            atomicAdd(&hsum[t], ssum[t]);
        }
    }
}

// cond(T): sum_{a<T} a <= (K - #{a>=T}) * T, exactly (T >= 1).
__device__ inline bool thresh_ok(unsigned long long F, unsigned long long C, int64_t K,
                                 unsigned long long T)
{
    if (T == 0) return false;
    if ((unsigned long long)K < C) return false;
    unsigned long long d = (unsigned long long)K - C;
    unsigned long long hi = __umul64hi(d, T), lo = d * T;
    return hi != 0 || lo >= F;
}

// One block of 256 threads: evaluate every bucket boundary, keep the least
// one that satisfies cond, descend into the bucket below it, clear the
// histogram for the next level.
__global__ void __launch_bounds__(256) k_mvs_radix_decide(SampleState *__restrict__ st, int64_t K,
                                                          unsigned long long *__restrict__ hcnt,
                                                          unsigned long long *__restrict__ hsum,
                                                          int32_t count_mode)
{
    __shared__ unsigned long long s_c[kDigitBuckets + 1], s_f[kDigitBuckets + 1];
    __shared__ int s_best;
    if (st->done) return;
    const int32_t nb = st->nbuckets;
    const int shift = st->shift;
    const unsigned long long lo = (unsigned long long)st->lo;
    // s_f[b] = F_below + the key sums of buckets below b; s_c[b] = C_above +
    // the counts of buckets b and above (b = 0..nb): each thread takes a run
    // of kPer buckets, the block scans the runs' totals
    constexpr int kPer = (kDigitBuckets + 255) / 256;
    __shared__ unsigned long long s_wf[4], s_wc[4];
    const int b0 = (int)threadIdx.x * kPer;
    unsigned long long cnt[kPer], sum[kPer], rf = 0, rc = 0;
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
        const int b = b0 + j;
        cnt[j] = b < nb ? hcnt[b] : 0ull;
        sum[j] = b < nb ? hsum[b] : 0ull;
        rf += sum[j];
        rc += cnt[j];
    }
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    const unsigned long long xf = wave_incl_sum(rf), xc = wave_incl_sum(rc);
    if (lane == 63) {
        s_wf[wid] = xf;
        s_wc[wid] = xc;
    }
    if (threadIdx.x == 0) s_best = nb + 1;
    __syncthreads();
    unsigned long long pf = xf - rf, pc = xc - rc, ctot = 0, ftot = 0;  // exclusive prefixes; totals
    for (int w = 0; w < 4; ++w) {
        if (w < wid) {
            pf += s_wf[w];
            pc += s_wc[w];
        }
        ctot += s_wc[w];
        ftot += s_wf[w];
    }
    const unsigned long long F0 = st->F_below, C0 = st->C_above;
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
        const int b = b0 + j;
        if (b <= nb) {
            s_f[b] = F0 + pf;
            s_c[b] = C0 + (ctot - pc);
        }
        pf += sum[j];
        pc += cnt[j];
    }
    // the boundary past the last bucket, when the runs end before it
    if (threadIdx.x == 0 && nb >= 256 * kPer) {
        s_f[nb] = F0 + ftot;
        s_c[nb] = C0;
    }
    __syncthreads();
    for (int b = threadIdx.x; b <= nb; b += blockDim.x) {
        unsigned long long T = lo + ((unsigned long long)b << shift);
        // count mode: the least T with fewer than K keys at or above it
        const bool ok = count_mode ? s_c[b] < (unsigned long long)K : thresh_ok(s_f[b], s_c[b], K, T);
        if (ok) atomicMin(&s_best, b);
    }
    __syncthreads();
    int best = s_best;
    if (threadIdx.x == 0) {
        if (best > nb || best == 0) {
            // cannot happen when the invariant holds; report instead of looping
            st->bad |= 2u;
            st->done = 1;
        } else if (shift == 0) {
            // count mode keeps the K-th largest key, one below that least T
            st->T = (long long)(lo + (unsigned long long)best) - (count_mode ? 1 : 0);
            st->done = 1;
        } else {
            st->F_below = s_f[best - 1];
            st->C_above = s_c[best];
            st->lo = (long long)(lo + ((unsigned long long)(best - 1) << shift));
            int ns = shift > kDigitBits ? shift - kDigitBits : 0;
            st->nbuckets = 1 << (shift - ns);
            st->shift = ns;
        }
    }
    for (int b = threadIdx.x; b < nb; b += blockDim.x) {
        hcnt[b] = 0;
        hsum[b] = 0;
    }
}

// Keep decision of every row; a block covers one compaction tile of 4096
// rows (16 per thread, a block stride apart) and writes its kept count.
template <int kSrc>
__global__ void __launch_bounds__(256) k_mvs_select(SampleSrc src, const int64_t *__restrict__ keys,
                                                    int64_t n, double lambda, SampleState *__restrict__ st,
                                                    uint64_t seed, uint64_t iteration,
                                                    int64_t row_offset, uint8_t *__restrict__ keep,
                                                    int32_t *__restrict__ tile_cnt, SampleRule rule,
                                                    ThreshFuse fuse)
{
    __shared__ int32_t red4[4];
    __shared__ unsigned long long s_T;
    const bool sgb = rule.mode == GBT_SAMPLE_SGB, goss = rule.mode == GBT_SAMPLE_GOSS;
    // SGB reads no key: every row's key stands at 0 below T = 1.  With the
    // threshold's first step fused, every block derives T from the key sums
    // and block 0 writes the state and the host flag (the other blocks read
    // none of the fields it writes).
    unsigned long long T;
    if (fuse.on) {
        if (threadIdx.x < 64) {
            const unsigned long long t = thresh_first_T_wave(st, fuse.K, fuse.check_log2n);
            if (threadIdx.x == 0) {
                s_T = t;
                if (blockIdx.x == 0) thresh_first(st, fuse.K, fuse.done_host, 0, fuse.check_log2n);
            }
        }
        __syncthreads();
        T = s_T;
    } else {
        T = sgb ? 1ull : (unsigned long long)st->T;
    }
    const int32_t e = st->e_key;
    const int64_t tbase = (int64_t)blockIdx.x * kCompactTile;
    // global row r draws word r mod 4 of the Philox block r div 4; when the
    // offset is a multiple of 4, a thread's four consecutive rows share one
    // block
    const bool aligned = (row_offset & 3) == 0;
    int32_t cnt = 0;
#pragma unroll 2
    for (int k = 0; k < kCompactTile / 1024; ++k) {
        const int64_t i0 = tbase + k * 1024 + 4 * (int64_t)threadIdx.x;
        if (i0 >= n) break;
        const bool full = i0 + 4 <= n;
        unsigned long long a[4] = {0, 0, 0, 0};
        if (sgb) {
        } else if (keys && full) {
            const longlong2 x = *(const longlong2 *)(keys + i0), y = *(const longlong2 *)(keys + i0 + 2);
            a[0] = (unsigned long long)x.x;
            a[1] = (unsigned long long)x.y;
            a[2] = (unsigned long long)y.x;
            a[3] = (unsigned long long)y.y;
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                a[j] = 0;
                if (i0 + j >= n) continue;
                if (keys) {
                    a[j] = (unsigned long long)keys[i0 + j];
                } else {
                    double g, h;
                    row_gh<kSrc>(src, i0 + j, &g, &h);
                    a[j] = (unsigned long long)(long long)rint(ldexp(mvs_r(g, h, lambda), e));
                }
            }
        }
        bool need = false;
#pragma unroll
        for (int j = 0; j < 4; ++j) need |= (i0 + j < n) && a[j] < T;
        need = need && !(rule.all_rest && !(rule.mode == GBT_SAMPLE_MVS));
        uint64_t U[4] = {0, 0, 0, 0};
        if (need) {
            const uint64_t g0 = (uint64_t)(row_offset + i0);
            uint64_t w[4];
            philox_block(g0 >> 2, iteration, seed, w);
            if (aligned) {
#pragma unroll
                for (int j = 0; j < 4; ++j) U[j] = w[j];
            } else {
                uint64_t w2[4];
                philox_block((g0 >> 2) + 1, iteration, seed, w2);
                const uint32_t s = (uint32_t)(g0 & 3);
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const uint32_t q = s + (uint32_t)j;  // 0..6: word q of the first block, else q - 4 of the next
                    U[j] = q == 0 ? w[0] : q == 1 ? w[1] : q == 2 ? w[2] : q == 3 ? w[3]
                         : q == 4 ? w2[0] : q == 5 ? w2[1] : w2[2];
                }
            }
        }
        uint32_t kb = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            if (i0 + j >= n) continue;
            const bool drawn = rule.all_rest || U[j] < rule.P;  // SGB, GOSS: the draw passes
            const bool kp = (sgb || goss) ? (!sgb && a[j] >= T) || drawn : a[j] >= T || __umul64hi(U[j], T) < a[j];
            kb |= (kp ? 1u : 0u) << (8 * j);
            cnt += kp ? 1 : 0;
        }
        if (full) {
            *(uint32_t *)(keep + i0) = kb;
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (i0 + j < n) keep[i0 + j] = (uint8_t)((kb >> (8 * j)) & 1u);
        }
    }
    cnt = wave_total(cnt);
    if ((threadIdx.x & 63) == 0) red4[threadIdx.x >> 6] = cnt;
    __syncthreads();
    if (threadIdx.x == 0 && tile_cnt) tile_cnt[blockIdx.x] = red4[0] + red4[1] + red4[2] + red4[3];
}

// f = 1: every row trains, unweighted.
__global__ void k_gw_all(const float2 *__restrict__ gpair, int64_t n, double2 *__restrict__ gw)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    float2 p = gpair[i];
    gw[i] = make_double2((double)p.x, (double)p.y);
}

// Compaction of one range of rows, tile by tile: the block rescans its tile's
// keep flags (exclusive, from the tile offset) into a list of the tile's
// kept rows; its threads then copy those rows into the sampled page
// together (16-byte pieces), and record each kept row's global id and
// reweighted pair, folding the maxima of |g'| and |h'|.
template <int kSrc>
__global__ void __launch_bounds__(256)
    k_compact_tiles(SampleSrc src, int64_t n, double lambda, SampleState *__restrict__ st,
                    const uint8_t *__restrict__ keep, const int32_t *__restrict__ tile_off,
                    int64_t tile0, int64_t row_lo, int64_t row_hi, const uint4 *__restrict__ words,
                    int32_t row_q4, uint4 *__restrict__ out_page, int32_t *__restrict__ sel,
                    double2 *__restrict__ gw, SampleRule rule, int64_t cap, int64_t self_tiles,
                    int32_t *__restrict__ total_host)
{
    __shared__ int32_t lds4[4];
    __shared__ unsigned long long red4[4];
    __shared__ uint16_t klist[kCompactTile];
    const int64_t tile = tile0 + blockIdx.x;
    const int64_t tbase = tile * kCompactTile;
    // self_tiles > 0: tile_off holds the selection's per-tile counts (no
    // scan ran); the block sums those before its tile, and block 0 all of
    // them for the host (the sample size)
    unsigned long long pre = 0, all = 0;
    if (self_tiles > 0) {
        for (int64_t k = threadIdx.x; k < tile; k += blockDim.x) pre += (unsigned long long)tile_off[k];
        if (blockIdx.x == 0)
            for (int64_t k = threadIdx.x; k < self_tiles; k += blockDim.x) all += (unsigned long long)tile_off[k];
    }
    const int64_t base = tbase + (int64_t)threadIdx.x * 16;
    uint32_t bits = 0;
    if (base + 16 <= n) {
        uint4 v = *(const uint4 *)(keep + base);
        uint32_t wv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int k = 0; k < 16; ++k) bits |= ((wv[k >> 2] >> (8 * (k & 3))) & 1u) << k;
    } else {
        for (int k = 0; k < 16; ++k)
            if (base + k < n && keep[base + k]) bits |= 1u << k;
    }
    // exclusive scan of the per-thread counts across the block
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    const int32_t cnt = __popc(bits);
    const int32_t x = wave_incl_sum(cnt);
    if (lane == 63) lds4[wid] = x;
    __syncthreads();
    int32_t run = x - cnt;
    for (int w = 0; w < wid; ++w) run += lds4[w];
    const int32_t nk = lds4[0] + lds4[1] + lds4[2] + lds4[3];
    while (bits) {
        const int k = __ffs(bits) - 1;
        bits &= bits - 1;
        klist[run++] = (uint16_t)(threadIdx.x * 16 + k);
    }
    __syncthreads();
    int64_t pos0;
    if (self_tiles > 0) {
        pos0 = (int64_t)block_sum_u64(pre, red4);
        if (blockIdx.x == 0) {
            all = block_sum_u64(all, red4);
            if (threadIdx.x == 0)
                __hip_atomic_store(total_host, (int32_t)all, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        }
    } else {
        pos0 = tile_off[tile];
    }
    if (pos0 + nk > cap) return;  // the whole block: the buffers are too small
    // the rows, 16 bytes per thread and step
    for (int32_t e = threadIdx.x; e < nk * row_q4; e += 256) {
        const int32_t j = e / row_q4, t = e - j * row_q4;
        const int64_t i = tbase + klist[j];
        if (i < row_lo || i >= row_hi) continue;
        out_page[(pos0 + j) * row_q4 + t] = words[(i - row_lo) * row_q4 + t];
    }
    // ids and reweighted pairs
    const unsigned long long T = (unsigned long long)st->T;
    const int32_t ek = st->e_key;
    unsigned long long mg = 0, mh = 0;
    for (int32_t j = threadIdx.x; j < nk; j += 256) {
        const int64_t i = tbase + klist[j];
        if (i < row_lo || i >= row_hi) continue;
        const int64_t pos = pos0 + j;
        sel[pos] = (int32_t)i;
        double g, h;
        row_gh<kSrc>(src, i, &g, &h);
        double w = 1.0;  // SGB
        if (rule.mode != GBT_SAMPLE_SGB) {
            unsigned long long a = (unsigned long long)(long long)rint(ldexp(mvs_r(g, h, lambda), ek));
            w = a >= T ? 1.0 : rule.mode == GBT_SAMPLE_GOSS ? rule.w_rest : (double)(long long)T / (double)(long long)a;
        }
        double2 v = make_double2(g * w, h * w);
        gw[pos] = v;
        unsigned long long bg = __double_as_longlong(fabs(v.x)), bh = __double_as_longlong(fabs(v.y));
        mg = bg > mg ? bg : mg;
        mh = bh > mh ? bh : mh;
    }
    mg = block_max_u64(mg, red4);
    mh = block_max_u64(mh, red4);
    if (threadIdx.x == 0) {
        if (mg) atomicMax(spread_at(st->gmax, blockIdx.x), mg);
        if (mh) atomicMax(spread_at(st->hmax, blockIdx.x), mh);
    }
}

// kSpec: also the keys' maximum and sum with the key exponent e_spec (the
// keys pass's, when e_spec turns out to be the exponent it would take).
template <bool kSpec>
__global__ void __launch_bounds__(256) k_gradients_rmax(int32_t loss, const float *__restrict__ margin,
                                                        const float *__restrict__ label, int64_t n,
                                                        float2 *__restrict__ gpair, double lambda,
                                                        SampleState *__restrict__ st, int32_t e_spec,
                                                        const int32_t *__restrict__ e_spec_at)
{
    __shared__ unsigned long long lds4[4];
    if (kSpec && e_spec_at) e_spec = *e_spec_at;
    unsigned long long b = 0, amx = 0, asm_ = 0;
    bool bad = false;
    auto one = [&](float m, float y, float2 *out) {
        double g, h;
        gradient_pair(loss, m, y, &g, &h);
        const float2 p = make_float2((float)g, (float)h);
        *out = p;
        const double x = mvs_r2((double)p.x, (double)p.y, lambda);
        bad |= !(x <= 1.7976931348623157e308);  // NaN or infinite
        const unsigned long long xb = __double_as_longlong(x);
        b = xb > b ? xb : b;
        if (kSpec) {
            const unsigned long long a = (unsigned long long)(long long)rint(ldexp(mvs_r((double)p.x, (double)p.y, lambda), e_spec));
            amx = a > amx ? a : amx;
            asm_ += a;
        }
    };
    const int64_t t0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x, step = (int64_t)gridDim.x * blockDim.x;
    if (((uintptr_t)margin & 7u) == 0 && ((uintptr_t)label & 7u) == 0 && ((uintptr_t)gpair & 15u) == 0) {
        // two rows per thread and step: 8-byte loads, one 16-byte store
        const int64_t np = n / 2;
        for (int64_t t = t0; t < np; t += step) {
            const float2 mv = ((const float2 *)margin)[t], lv = ((const float2 *)label)[t];
            float2 p0, p1;
            one(mv.x, lv.x, &p0);
            one(mv.y, lv.y, &p1);
            ((float4 *)gpair)[t] = make_float4(p0.x, p0.y, p1.x, p1.y);
        }
        if ((n & 1) && t0 == 0) one(margin[n - 1], label[n - 1], &gpair[n - 1]);
    } else {
        for (int64_t i = t0; i < n; i += step) one(margin[i], label[i], &gpair[i]);
    }
    if (bad) atomicOr(&st->bad, 1u);
    b = block_max_u64(b, lds4);
    if (threadIdx.x == 0 && b) atomicMax(spread_at(st->rmax, blockIdx.x), b);
    if (kSpec) {
        amx = block_max_u64(amx, lds4);
        asm_ = block_sum_u64(asm_, lds4);
        if (threadIdx.x == 0) {
            if (amx) atomicMax(spread_at(st->amax, blockIdx.x), amx);
            if (asm_) atomicAdd(spread_at(st->asum, blockIdx.x), asm_);
            if (blockIdx.x == 0) st->e_key = e_spec;
        }
    }
}

// The keys' maximum and sum cleared (a speculated exponent was wrong).
__global__ void k_keys_reset(SampleState *__restrict__ st)
{
    for (int t = threadIdx.x; t < kSpread * kLineWords; t += blockDim.x) {
        (&st->amax[0][0])[t] = 0ull;
        (&st->asum[0][0])[t] = 0ull;
    }
}

// The maxima of |g'| and |h'| cleared (a compaction is redone).
__global__ void k_fx_max_reset(SampleState *__restrict__ st)
{
    for (int t = threadIdx.x; t < kSpread * kLineWords; t += blockDim.x) {
        (&st->gmax[0][0])[t] = 0ull;
        (&st->hmax[0][0])[t] = 0ull;
    }
}

// ------------------------------------------------------------ fixed point
__global__ void __launch_bounds__(256) k_fx_max(const double2 *__restrict__ gw, int64_t R,
                                                SampleState *__restrict__ st)
{
    __shared__ unsigned long long lds4[4];
    unsigned long long bg = 0, bh = 0;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < R;
         i += (int64_t)gridDim.x * blockDim.x) {
        double2 v = gw[i];
        unsigned long long a = __double_as_longlong(fabs(v.x)), b = __double_as_longlong(fabs(v.y));
        bg = a > bg ? a : bg;
        bh = b > bh ? b : bh;
    }
    bg = block_max_u64(bg, lds4);
    bh = block_max_u64(bh, lds4);
    if (threadIdx.x == 0) {
        if (bg) atomicMax(spread_at(st->gmax, blockIdx.x), bg);
        if (bh) atomicMax(spread_at(st->hmax, blockIdx.x), bh);
    }
}

// q = rint((g', h') * 2^(e_g, e_h)), e = 62 - E - ceil(log2 R); also the
// root sums (integer, order independent).
__global__ void __launch_bounds__(256) k_fx_convert(const double2 *__restrict__ gw, int64_t R,
                                                    int32_t log2R, SampleState *__restrict__ st,
                                                    longlong2 *__restrict__ q)
{
    __shared__ unsigned long long lds4[4], m2[2];
    int Eg, Eh;
    frexp(__longlong_as_double(block_fold_max(st->gmax, &m2[0])), &Eg);
    frexp(__longlong_as_double(block_fold_max(st->hmax, &m2[1])), &Eh);
    const int32_t eg = 62 - Eg - log2R, eh = 62 - Eh - log2R;
    unsigned long long sg = 0, sh = 0;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < R;
         i += (int64_t)gridDim.x * blockDim.x) {
        double2 v = gw[i];
        long long qg = (long long)rint(ldexp(v.x, eg)), qh = (long long)rint(ldexp(v.y, eh));
        q[i] = make_longlong2(qg, qh);
        sg += (unsigned long long)qg;
        sh += (unsigned long long)qh;
    }
    sg = block_sum_u64(sg, lds4);
    sh = block_sum_u64(sh, lds4);
    if (threadIdx.x == 0) {
        if (sg) atomicAdd(spread_at(st->root_g, blockIdx.x), sg);
        if (sh) atomicAdd(spread_at(st->root_h, blockIdx.x), sh);
        if (blockIdx.x == 0) {
            st->e_g = eg;
            st->e_h = eh;
        }
    }
}

// The MVS lambda estimate's two passes over every row, with the pair
// recomputed from margin and label each time and rounded to float as
// gbt_gradients stores it (nothing per row is kept): pass 0 folds the
// maxima of |g| and |h|, pass 1 converts to the fixed point of those
// maxima and folds the exact integer sums.
template <int kPass>
__global__ void __launch_bounds__(256) k_lambda_pass(int32_t loss, const float *__restrict__ margin,
                                                     const float *__restrict__ label, int64_t n, int32_t log2n,
                                                     SampleState *__restrict__ st)
{
    __shared__ unsigned long long lds4[4], m2[2];
    int32_t eg = 0, eh = 0;
    if (kPass == 1) {
        int Eg, Eh;
        frexp(__longlong_as_double(block_fold_max(st->gmax, &m2[0])), &Eg);
        frexp(__longlong_as_double(block_fold_max(st->hmax, &m2[1])), &Eh);
        eg = 62 - Eg - log2n;
        eh = 62 - Eh - log2n;
    }
    unsigned long long a = 0, b = 0;
    bool bad = false;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        double g, h;
        gradient_pair(loss, margin[i], label[i], &g, &h);
        const double gf = (double)(float)g, hf = (double)(float)h;
        if (kPass == 0) {
            bad |= !(fabs(gf) <= 1.7976931348623157e308) || !(fabs(hf) <= 1.7976931348623157e308);
            const unsigned long long x = __double_as_longlong(fabs(gf)), y = __double_as_longlong(fabs(hf));
            a = x > a ? x : a;
            b = y > b ? y : b;
        } else {
            a += (unsigned long long)(long long)rint(ldexp(gf, eg));
            b += (unsigned long long)(long long)rint(ldexp(hf, eh));
        }
    }
    if (kPass == 0) {
        if (bad) atomicOr(&st->bad, 1u);
        a = block_max_u64(a, lds4);
        b = block_max_u64(b, lds4);
        if (threadIdx.x == 0) {
            if (a) atomicMax(spread_at(st->gmax, blockIdx.x), a);
            if (b) atomicMax(spread_at(st->hmax, blockIdx.x), b);
        }
    } else {
        a = block_sum_u64(a, lds4);
        b = block_sum_u64(b, lds4);
        if (threadIdx.x == 0) {
            if (a) atomicAdd(spread_at(st->root_g, blockIdx.x), a);
            if (b) atomicAdd(spread_at(st->root_h, blockIdx.x), b);
            if (blockIdx.x == 0) {
                st->e_g = eg;
                st->e_h = eh;
            }
        }
    }
}

__global__ void k_state_init(SampleState *st) { state_reset_block(st); }

__global__ void k_zero_u64(unsigned long long *p, int64_t n)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0ull;
}

static unsigned blocks(int64_t n, int t = 256) { return (unsigned)((n + t - 1) / t); }

static unsigned rblocks(int64_t n) { return std::max(1u, std::min(blocks(n), (unsigned)kReduceGrid)); }

static int32_t log2_ceil(int64_t v) { return v <= 1 ? 0 : ceil_log2_u64((uint64_t)v); }

// ------------------------------------------------------------ drivers
gbt_status wait_flag(gbt_ctx *c, volatile int32_t *done_poll)
{
    const auto t0 = std::chrono::steady_clock::now();
    for (uint32_t spin = 0; *done_poll < 0; ++spin) {
        if ((spin & 1023u) == 0 && std::chrono::steady_clock::now() - t0 > std::chrono::seconds(2)) {
            GBT_HIP(hipStreamSynchronize(c->stream));  // the flag is written by then
            break;
        }
    }
    return GBT_OK;
}

namespace {

void keys_pass(gbt_ctx *c, const SampleSrc &src, int kind, const int64_t *keys, int64_t n, double lambda,
               int32_t l2, SampleState *st)
{
    if (kind == kSrcGpair)
        k_mvs_keys<kSrcGpair><<<rblocks(n), 256, 0, c->stream>>>(src, n, lambda, l2, st, (int64_t *)keys);
    else
        k_mvs_keys<kSrcMargin><<<rblocks(n), 256, 0, c->stream>>>(src, n, lambda, l2, st, (int64_t *)keys);
}


// After the threshold's first kernel: with a host flag, its outcome (1 the
// closed form holds, 0 a descent is needed, 2 the guessed key exponent was
// wrong: the keys pass and the first kernel again); then the radix descent
// unless the closed form held.
gbt_status threshold_rest(gbt_ctx *c, const SampleSrc &src, int kind, const int64_t *keys, int64_t n,
                          double lambda, int64_t K, SampleState *st, bool count_mode, volatile int32_t *done_poll,
                          int32_t *done_dev)
{
    const int32_t l2 = log2_ceil(n);
    if (done_poll) {
        GBT_TRY(wait_flag(c, done_poll));
        if (*done_poll == 2) {
            // the guessed exponent was not the keys': the keys pass after all
            k_keys_reset<<<1, 256, 0, c->stream>>>(st);
            GBT_LAUNCHED();
            keys_pass(c, src, kind, keys, n, lambda, l2, st);
            GBT_LAUNCHED();
            *done_poll = -1;
            k_mvs_thresh_init<<<1, 64, 0, c->stream>>>(st, K, done_dev, count_mode ? 1 : 0, -1);
            GBT_LAUNCHED();
            GBT_TRY(wait_flag(c, done_poll));
        }
        if (*done_poll == 1) return GBT_OK;
    }
    unsigned long long *hist = nullptr;
    GBT_TRY(scratch_t(c, kScrMisc, 2 * kDigitBuckets, &hist));
    k_zero_u64<<<blocks(2 * kDigitBuckets), 256, 0, c->stream>>>(hist, 2 * kDigitBuckets);
    GBT_LAUNCHED();
    // Every key is at most 2^(62 - ceil(log2 n)), so the descent needs at
    // most ceil((63 - ceil(log2 n)) / 11) levels; levels past the answer (or
    // past the closed form) return at once.
    const int levels = std::max(1, (63 - l2 + kDigitBits - 1) / kDigitBits);
    unsigned grid = (unsigned)std::min<int64_t>(std::max<int64_t>(blocks(n), 1), 2 * kCUs);
    for (int lev = 0; lev < levels; ++lev) {
        if (kind == kSrcGpair)
            k_mvs_radix_hist<kSrcGpair><<<grid, 256, 0, c->stream>>>(src, keys, n, lambda, l2, st, hist,
                                                                     hist + kDigitBuckets);
        else
            k_mvs_radix_hist<kSrcMargin><<<grid, 256, 0, c->stream>>>(src, keys, n, lambda, l2, st, hist,
                                                                      hist + kDigitBuckets);
        GBT_LAUNCHED();
        k_mvs_radix_decide<<<1, 256, 0, c->stream>>>(st, K, hist, hist + kDigitBuckets, count_mode ? 1 : 0);
        GBT_LAUNCHED();
    }
    return GBT_OK;
}

}  // namespace

gbt_status mvs_threshold(gbt_ctx *c, const SampleSrc &src, int kind, const int64_t *keys, int64_t n,
                         double lambda, int64_t K, SampleState *st, bool skip_closed, bool rmax_done,
                         bool count_mode, bool keys_spec, bool defer, ThreshFuse *fuse)
{
    GBT_CHECK(!fuse || (defer && !count_mode), "a threshold fused into the selection is deferred MVS");
    GBT_CHECK(!keys_spec || (skip_closed && rmax_done && !keys && !count_mode),
              "speculated key sums need the host's closed-form test");
    GBT_CHECK(!defer || skip_closed, "a deferred threshold needs the host's closed-form test");
    const int32_t l2 = log2_ceil(n);
    if (n > 0) {
        if (rmax_done)
            ;
        else if (kind == kSrcGpair)
            k_mvs_rmax<kSrcGpair><<<rblocks(n), 256, 0, c->stream>>>(src, n, lambda, st);
        else
            k_mvs_rmax<kSrcMargin><<<rblocks(n), 256, 0, c->stream>>>(src, n, lambda, st);
        GBT_LAUNCHED();
    }
    // speculated: the gradient pass summed the keys with a guessed exponent
    if (n > 0 && !keys_spec) {
        keys_pass(c, src, kind, keys, n, lambda, l2, st);
        GBT_LAUNCHED();
    }
    // skip_closed: the host learns from pinned memory whether the closed form
    // holds (it waits for the passes above, nothing else is queued) and then
    // launches no descent levels, which would all return at once
    volatile int32_t *done_poll = nullptr;
    int32_t *done_dev = nullptr;
    if (skip_closed) {
        void *hio, *hio_d;
        GBT_TRY(host_io(c, 64, &hio, &hio_d));
        done_poll = (volatile int32_t *)hio;
        done_dev = (int32_t *)hio_d;
        *done_poll = -1;
    }
    if (fuse) {
        *fuse = ThreshFuse{K, done_dev, keys_spec && n > 0 ? l2 : -1, 1};
        return GBT_OK;
    }
    k_mvs_thresh_init<<<1, 64, 0, c->stream>>>(st, K, done_dev, count_mode ? 1 : 0, keys_spec && n > 0 ? l2 : -1);
    GBT_LAUNCHED();
    if (defer) return GBT_OK;
    return threshold_rest(c, src, kind, keys, n, lambda, K, st, count_mode, done_poll, done_dev);
}

gbt_status mvs_threshold_resume(gbt_ctx *c, const SampleSrc &src, int kind, const int64_t *keys, int64_t n,
                                double lambda, int64_t K, SampleState *st, bool *redo)
{
    void *hio, *hio_d;
    GBT_TRY(host_io(c, 64, &hio, &hio_d));
    volatile int32_t *done_poll = (volatile int32_t *)hio;
    GBT_TRY(wait_flag(c, done_poll));
    *redo = *done_poll != 1;
    if (!*redo) return GBT_OK;
    return threshold_rest(c, src, kind, keys, n, lambda, K, st, false, done_poll, (int32_t *)hio_d);
}

gbt_status mvs_select(gbt_ctx *c, const SampleSrc &src, int kind, const int64_t *keys, int64_t n,
                      double lambda, SampleState *st, uint64_t seed, uint64_t iteration,
                      int64_t row_offset, uint8_t *keep, int32_t *tile_cnt, const SampleRule &rule,
                      const ThreshFuse &fuse)
{
    GBT_CHECK(!fuse.on || rule.mode == GBT_SAMPLE_MVS, "a fused threshold needs the MVS rule");
    if (n == 0) return GBT_OK;
    const unsigned grid = (unsigned)((n + kCompactTile - 1) / kCompactTile);
    if (kind == kSrcGpair)
        k_mvs_select<kSrcGpair><<<grid, 256, 0, c->stream>>>(src, keys, n, lambda, st, seed, iteration,
                                                             row_offset, keep, tile_cnt, rule, fuse);
    else
        k_mvs_select<kSrcMargin><<<grid, 256, 0, c->stream>>>(src, keys, n, lambda, st, seed, iteration,
                                                              row_offset, keep, tile_cnt, rule, fuse);
    GBT_LAUNCHED();
    return GBT_OK;
}

gbt_status gw_all(gbt_ctx *c, const float *gpair, int64_t n, double *gw)
{
    if (n == 0) return GBT_OK;
    k_gw_all<<<blocks(n), 256, 0, c->stream>>>((const float2 *)gpair, n, (double2 *)gw);
    GBT_LAUNCHED();
    return GBT_OK;
}

gbt_status gradients_rmax(gbt_ctx *c, int32_t loss, const float *margin, const float *label, int64_t n,
                          float *gpair, double lambda, SampleState *st, int32_t e_spec,
                          const int32_t *e_spec_at)
{
    if (n == 0) return GBT_OK;
    if (e_spec == kNoKeySpec && !e_spec_at)
        k_gradients_rmax<false><<<rblocks(n), 256, 0, c->stream>>>(loss, margin, label, n, (float2 *)gpair, lambda,
                                                                   st, 0, nullptr);
    else
        k_gradients_rmax<true><<<rblocks(n), 256, 0, c->stream>>>(loss, margin, label, n, (float2 *)gpair, lambda,
                                                                  st, e_spec, e_spec_at);
    GBT_LAUNCHED();
    return GBT_OK;
}

gbt_status keep_tile_offsets(gbt_ctx *c, int64_t n, int32_t *tile_off, int32_t *total_host)
{
    return scan_tile_counts(c, tile_off, (n + kCompactTile - 1) / kCompactTile, total_host);
}

gbt_status mvs_compact_tiles(gbt_ctx *c, const SampleSrc &src, int kind, int64_t n, double lambda,
                             SampleState *st, const uint8_t *keep, const int32_t *tile_off,
                             int64_t row_lo, int64_t row_hi, const uint32_t *words, int32_t row_words,
                             uint32_t *out_page, int32_t *sel, double *gw, const SampleRule &rule, int64_t cap,
                             int32_t *total_host)
{
    if (row_hi <= row_lo) return GBT_OK;
    const int64_t t0 = row_lo / kCompactTile, t1 = (row_hi - 1) / kCompactTile + 1;
    const unsigned grid = (unsigned)(t1 - t0);
    // total_host: the offsets come from the counts (all of rows [0, n))
    GBT_CHECK(!total_host || (row_lo == 0 && row_hi == n), "a compaction that sums its own tile offsets covers every row");
    const int64_t self_tiles = total_host ? (int64_t)grid : 0;
    if (kind == kSrcGpair)
        k_compact_tiles<kSrcGpair><<<grid, 256, 0, c->stream>>>(
            src, n, lambda, st, keep, tile_off, t0, row_lo, row_hi, (const uint4 *)words, row_words / 4,
            (uint4 *)out_page, sel, (double2 *)gw, rule, cap, self_tiles, total_host);
    else
        k_compact_tiles<kSrcMargin><<<grid, 256, 0, c->stream>>>(
            src, n, lambda, st, keep, tile_off, t0, row_lo, row_hi, (const uint4 *)words, row_words / 4,
            (uint4 *)out_page, sel, (double2 *)gw, rule, cap, self_tiles, total_host);
    GBT_LAUNCHED();
    return GBT_OK;
}

gbt_status fx_max_reset(gbt_ctx *c, SampleState *st)
{
    k_fx_max_reset<<<1, 256, 0, c->stream>>>(st);
    GBT_LAUNCHED();
    return GBT_OK;
}

gbt_status fixed_point(gbt_ctx *c, const double *gw, int64_t R, SampleState *st, int64_t *q, bool fx_max_done)
{
    if (R == 0) {
        k_fx_convert<<<1, 256, 0, c->stream>>>((const double2 *)gw, 0, 0, st, (longlong2 *)q);
        GBT_LAUNCHED();
        return GBT_OK;
    }
    if (!fx_max_done) {
        k_fx_max<<<rblocks(R), 256, 0, c->stream>>>((const double2 *)gw, R, st);
        GBT_LAUNCHED();
    }
    k_fx_convert<<<rblocks(R), 256, 0, c->stream>>>((const double2 *)gw, R, log2_ceil(R), st,
                                                   (longlong2 *)q);
    GBT_LAUNCHED();
    return GBT_OK;
}

gbt_status lambda_sums(gbt_ctx *c, int32_t loss, const float *margin, const float *label, int64_t n,
                       SampleState *st)
{
    if (n == 0) return GBT_OK;
    k_lambda_pass<0><<<rblocks(n), 256, 0, c->stream>>>(loss, margin, label, n, 0, st);
    GBT_LAUNCHED();
    k_lambda_pass<1><<<rblocks(n), 256, 0, c->stream>>>(loss, margin, label, n, log2_ceil(n), st);
    GBT_LAUNCHED();
    return GBT_OK;
}

gbt_status state_init(gbt_ctx *c, SampleState *st)
{
    k_state_init<<<1, 256, 0, c->stream>>>(st);
    GBT_LAUNCHED();
    return GBT_OK;
}

}  // namespace gbt
