// quantize.hip -- Sec. 2.2 and Sec. 3.1/3.2 of the paper: exact quantile cuts
// over a sketch sample (Alg. 2/3) and bit-packed ELLPACK pages (Alg. 4/5).
//
// Cuts: for a feature with sorted non-missing sketch values s_0..s_{N-1}
// and B = max_bin, candidate k = s[ceil(kN/B)-1] (k = 1..B-1), duplicates
// and values >= s_{N-1} dropped.  The order statistics are found on the GPU
// by a multi-way bisection over order-preserving 32-bit keys: each pass
// splits every unresolved target's key interval into 16 parts and counts,
// per feature, the keys at or below every split point (LDS counters, one
// binary search per key).  Eight passes resolve 32 bits.  The host only
// narrows the intervals from the tiny count tables.
//
// Pages: row-major rows of row_words 32-bit words; a row is the LSB-first
// bit stream of its stride symbols (w bits each), zero padded.
#include "common.h"
#include "hist_impl.h"
#include "sketch_impl.h"

#include <algorithm>
#include <cerrno>
#include <cstring>
#include <fcntl.h>
#include <unistd.h>

using namespace gbt;

namespace {

constexpr uint32_t kNanKey = 0xffffffffu;
constexpr uint32_t kMaxKey = 0xff7fffffu;  // key of the largest finite float
constexpr int kBisectWays = 16;            // parts per interval per pass
constexpr int kLdsBounds = 4096;           // split points held in LDS

__device__ __host__ inline uint32_t float_key(float x)
{
    uint32_t u;
    if (x == 0.0f) x = 0.0f;  // -0 -> +0
    memcpy(&u, &x, 4);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

inline float key_float(uint32_t k)
{
    uint32_t u = (k & 0x80000000u) ? (k & 0x7fffffffu) : ~k;
    float x;
    memcpy(&x, &u, 4);
    return x;
}

enum { kStNan = 0, kStInf, kStMaxNnz, kStKeys, kStBadIndex, kStWords };

// Dense batch: validate every value, record the sketch keys of the sampled
// rows (global row g with g % stride == 0) feature-major: sample g / stride
// at column g / stride - s_base of a key matrix of n_sketch columns.
__global__ void k_dense_sketch(const float *__restrict__ X, int64_t rows, int32_t m, int64_t ld,
                               int64_t row0, int64_t stride, int64_t n_sketch, int64_t s_base,
                               uint32_t *__restrict__ keys, unsigned long long *__restrict__ st)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    bool nan = false, inf = false;
    if (i < rows) {
        int64_t g = row0 + i;
        bool take = (g % stride) == 0;
        int64_t s = g / stride - s_base;
        const float *x = X + i * ld;
        for (int32_t j = 0; j < m; ++j) {
            float v = x[j];
            bool isn = v != v;
            nan |= isn;
            inf |= (!isn && (v - v) != 0.0f);
            if (take && s >= 0 && s < n_sketch) keys[(int64_t)j * n_sketch + s] = isn ? kNanKey : float_key(v);
        }
    }
    if (__any(nan) && (threadIdx.x & 63) == 0) atomicOr(&st[kStNan], 1ull);
    if (__any(inf) && (threadIdx.x & 63) == 0) atomicOr(&st[kStInf], 1ull);
}

// CSR batch: validate indices, count present (non-NaN) entries per row, and
// append the (feature, key) pairs of sampled rows.
__global__ void k_csr_sketch(const int64_t *__restrict__ indptr, const int32_t *__restrict__ idx,
                             const float *__restrict__ val, int64_t rows, int32_t m, int64_t row0,
                             int64_t stride, uint32_t *__restrict__ keys,
                             int32_t *__restrict__ feats, unsigned long long *__restrict__ st)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= rows) return;
    int64_t base = indptr[0];
    int64_t e0 = indptr[i] - base, e1 = indptr[i + 1] - base;
    int32_t prev = -1, cnt = 0;
    bool inf = false, bad = e1 < e0;
    for (int64_t e = e0; e < e1; ++e) {
        int32_t j = idx[e];
        float v = val[e];
        if (j <= prev || j >= m) bad = true;
        prev = j;
        bool isn = v != v;
        inf |= (!isn && (v - v) != 0.0f);
        cnt += !isn;
    }
    if (bad) atomicOr(&st[kStBadIndex], 1ull);
    if (inf) atomicOr(&st[kStInf], 1ull);
    atomicMax(&st[kStMaxNnz], (unsigned long long)cnt);
    if (bad || ((row0 + i) % stride) != 0 || cnt == 0) return;
    unsigned long long at = atomicAdd(&st[kStKeys], (unsigned long long)cnt);
    for (int64_t e = e0; e < e1; ++e) {
        float v = val[e];
        if (v != v) continue;
        keys[at] = float_key(v);
        feats[at] = idx[e];
        ++at;
    }
}

__global__ void k_feat_count(const int32_t *__restrict__ feats, int64_t n,
                             unsigned long long *__restrict__ cnt)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) atomicAdd(&cnt[feats[i]], 1ull);
}

__global__ void k_feat_scatter(const int32_t *__restrict__ feats, const uint32_t *__restrict__ keys,
                               int64_t n, unsigned long long *__restrict__ cursor,
                               uint32_t *__restrict__ out)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) out[atomicAdd(&cursor[feats[i]], 1ull)] = keys[i];
}

// One work item: keys[begin, end) of feature `feat`; its split points are
// bounds[boff[feat] .. boff[feat+1]) (sorted, distinct).  cnt[boff[f] + t]
// receives the number of keys k with bounds[t-1] < k <= bounds[t].
struct CountWork {
    int64_t begin, end;
    int32_t feat;
    int32_t pad0;
};

template <bool kLds>
__global__ void __launch_bounds__(256) k_bisect_count(const uint32_t *__restrict__ keys,
                                                      const CountWork *__restrict__ work,
                                                      const uint32_t *__restrict__ bounds,
                                                      const int32_t *__restrict__ boff,
                                                      unsigned int *__restrict__ cnt)
{
    __shared__ uint32_t sb[kLds ? kLdsBounds : 1];
    __shared__ unsigned int sc[kLds ? kLdsBounds : 1];
    CountWork wk = work[blockIdx.x];
    int32_t b0 = boff[wk.feat], nb = boff[wk.feat + 1] - b0;
    const uint32_t *bd = bounds + b0;
    if (kLds) {
        for (int t = threadIdx.x; t < nb; t += blockDim.x) {
            sb[t] = bd[t];
            sc[t] = 0;
        }
        __syncthreads();
    }
    for (int64_t i = wk.begin + threadIdx.x; i < wk.end; i += blockDim.x) {
        uint32_t k = keys[i];
        if (k == kNanKey) continue;
        // first split point >= k
        int32_t lo = 0, hi = nb;
        while (lo < hi) {
            int32_t mid = (lo + hi) >> 1;
            uint32_t b = kLds ? sb[mid] : bd[mid];
            if (b < k)
                lo = mid + 1;
            else
                hi = mid;
        }
        if (lo < nb) {
            if (kLds)
                atomicAdd(&sc[lo], 1u);
            else
                atomicAdd(&cnt[b0 + lo], 1u);
        }
    }
    if (kLds) {
        __syncthreads();
        for (int t = threadIdx.x; t < nb; t += blockDim.x)
            if (sc[t]) atomicAdd(&cnt[b0 + t], sc[t]);
    }
}

__device__ inline int32_t lookup_bin(const float *__restrict__ cuts, int32_t nc, float x)
{
    int32_t lo = 0, hi = nc;
    while (lo < hi) {
        int32_t mid = (lo + hi) >> 1;
        if (cuts[mid] < x)
            lo = mid + 1;
        else
            hi = mid;
    }
    return lo;
}

struct BitWriter {
    uint32_t *out;
    uint64_t acc = 0;
    int32_t nbits = 0, k = 0;
    __device__ BitWriter(uint32_t *o) : out(o) {}
    __device__ void put(uint32_t sym, int32_t w)
    {
        acc |= (uint64_t)sym << nbits;
        nbits += w;
        while (nbits >= 32) {
            out[k++] = (uint32_t)acc;
            acc >>= 32;
            nbits -= 32;
        }
    }
    __device__ void finish(int32_t row_words)
    {
        if (nbits > 0) out[k++] = (uint32_t)acc;
        while (k < row_words) out[k++] = 0u;
    }
};

__global__ void k_encode_dense(const float *__restrict__ X, int64_t rows, int32_t m, int64_t ld,
                               const int32_t *__restrict__ cut_ptr,
                               const float *__restrict__ cut_values, int32_t w, int32_t row_words,
                               uint32_t null_sym, uint32_t *__restrict__ out)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= rows) return;
    const float *x = X + i * ld;
    BitWriter bw(out + i * row_words);
    for (int32_t j = 0; j < m; ++j) {
        float v = x[j];
        uint32_t sym;
        if (v != v) {
            sym = null_sym;
        } else {
            int32_t c0 = cut_ptr[j];
            sym = (uint32_t)lookup_bin(cut_values + c0, cut_ptr[j + 1] - c0, v);
        }
        bw.put(sym, w);
    }
    bw.finish(row_words);
}

__global__ void k_encode_csr(const int64_t *__restrict__ indptr, const int32_t *__restrict__ idx,
                             const float *__restrict__ val, int64_t rows,
                             const int32_t *__restrict__ cut_ptr,
                             const float *__restrict__ cut_values,
                             const int32_t *__restrict__ bin_ptr, int32_t w, int32_t stride,
                             int32_t row_words, uint32_t null_sym, uint32_t *__restrict__ out,
                             unsigned long long *__restrict__ st)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= rows) return;
    int64_t base = indptr[0];
    int64_t e0 = indptr[i] - base, e1 = indptr[i + 1] - base;
    BitWriter bw(out + i * row_words);
    int32_t s = 0;
    for (int64_t e = e0; e < e1; ++e) {
        float v = val[e];
        if (v != v) continue;
        if (s >= stride) {  // more entries than the sketch pass saw in any row
            atomicOr(&st[kStBadIndex], 1ull);
            break;
        }
        int32_t j = idx[e];
        int32_t c0 = cut_ptr[j];
        bw.put((uint32_t)bin_ptr[j] + (uint32_t)lookup_bin(cut_values + c0, cut_ptr[j + 1] - c0, v),
               w);
        ++s;
    }
    for (; s < stride; ++s) bw.put(null_sym, w);
    bw.finish(row_words);
}

unsigned grid_for(int64_t n, int threads) { return (unsigned)((n + threads - 1) / threads); }

}  // namespace

// ------------------------------------------------------------------ quantizer
struct gbt_quantizer {
    gbt_ctx *ctx = nullptr;
    gbt_quant_params p{};
    int32_t m = 0;
    int32_t kind = GBT_INPUT_DENSE_F32;
    int64_t n_total = 0;
    int64_t stride = 1;
    int64_t n_sketch = 0;            // dense: sketch rows
    uint32_t *keys = nullptr;        // dense: m*n_sketch; CSR: appended pairs
    size_t keys_bytes = 0;
    int32_t *feats = nullptr;        // CSR only
    size_t feats_bytes = 0;
    int64_t keys_cap = 0;
    unsigned long long *st = nullptr;  // device status words
    int64_t sketched_rows = 0;
    int64_t encoded_rows = 0;
    bool cuts_done = false;
    gbt_matrix *mat = nullptr;
    // staging of host batches
    void *stage = nullptr;
    size_t stage_bytes = 0;
    uint32_t *enc = nullptr;         // encoded rows of one batch
    size_t enc_bytes = 0;
    // disk pages: their directory, and a pinned buffer the encoded rows
    // pass through on their way to the files
    std::string dir;
    void *bounce = nullptr;
    size_t bounce_bytes = 0;
    // merged sketch (sketch_summary > 0): the running summaries, and the
    // keys of one batch
    MergeSketch *ms = nullptr;
    uint32_t *bkeys = nullptr;
    size_t bkeys_bytes = 0;
};

namespace {

gbt_status ensure_buf(gbt_ctx *c, void **p, size_t *have, size_t want)
{
    if (*have >= want) return GBT_OK;
    GBT_HIP(hipStreamSynchronize(c->stream));
    dev_free(c, *p, *have);
    *p = nullptr;
    *have = 0;
    GBT_TRY(dev_alloc(c, want, p));
    *have = want;
    return GBT_OK;
}

// Device views of a batch (host batches are copied to the staging buffer).
struct DevBatch {
    const float *values = nullptr;
    const int64_t *indptr = nullptr;
    const int32_t *indices = nullptr;
    int64_t rows = 0, ld = 0, nnz = 0;
};

gbt_status stage_batch(gbt_quantizer *q, const gbt_input *in, DevBatch *b)
{
    gbt_ctx *c = q->ctx;
    GBT_CHECK(in, "batch is NULL");
    GBT_CHECK(in->kind == q->kind, "batch kind %d differs from the quantizer's %d", in->kind,
              q->kind);
    GBT_CHECK(in->n_cols == q->m, "batch has %d columns, expected %d", in->n_cols, q->m);
    GBT_CHECK(in->n_rows >= 0, "negative row count");
    b->rows = in->n_rows;
    if (in->kind == GBT_INPUT_DENSE_F32) {
        GBT_CHECK(in->ld >= in->n_cols, "ld %lld < n_cols %d", (long long)in->ld, in->n_cols);
        GBT_CHECK(in->values || in->n_rows == 0, "dense values are NULL");
        b->ld = in->ld;
        if (in->location == GBT_LOC_DEVICE) {
            b->values = in->values;
            return GBT_OK;
        }
        size_t bytes = (size_t)in->n_rows * (size_t)in->ld * sizeof(float);
        GBT_TRY(ensure_buf(c, &q->stage, &q->stage_bytes, bytes));
        if (bytes)
            GBT_HIP(hipMemcpyAsync(q->stage, in->values, bytes, hipMemcpyHostToDevice, c->stream));
        b->values = (const float *)q->stage;
        return GBT_OK;
    }
    GBT_CHECK(in->indptr, "CSR indptr is NULL");
    GBT_CHECK(in->nnz >= 0, "negative nnz");
    b->nnz = in->nnz;
    if (in->location == GBT_LOC_DEVICE) {
        b->values = in->values;
        b->indptr = in->indptr;
        b->indices = in->indices;
        return GBT_OK;
    }
    GBT_CHECK(in->indptr[in->n_rows] - in->indptr[0] == in->nnz,
              "CSR indptr spans %lld entries but nnz is %lld",
              (long long)(in->indptr[in->n_rows] - in->indptr[0]), (long long)in->nnz);
    size_t b_ip = (size_t)(in->n_rows + 1) * 8, b_ix = (size_t)in->nnz * 4, b_v = b_ix;
    size_t o_ix = (b_ip + 255) / 256 * 256, o_v = o_ix + (b_ix + 255) / 256 * 256;
    GBT_TRY(ensure_buf(c, &q->stage, &q->stage_bytes, o_v + b_v + 256));
    char *s = (char *)q->stage;
    GBT_HIP(hipMemcpyAsync(s, in->indptr, b_ip, hipMemcpyHostToDevice, c->stream));
    if (b_ix) {
        GBT_HIP(hipMemcpyAsync(s + o_ix, in->indices, b_ix, hipMemcpyHostToDevice, c->stream));
        GBT_HIP(hipMemcpyAsync(s + o_v, in->values, b_v, hipMemcpyHostToDevice, c->stream));
    }
    b->indptr = (const int64_t *)s;
    b->indices = (const int32_t *)(s + o_ix);
    b->values = (const float *)(s + o_v);
    return GBT_OK;
}

gbt_status read_status(gbt_quantizer *q, unsigned long long *out)
{
    GBT_HIP(hipMemcpyAsync(out, q->st, kStWords * sizeof(unsigned long long), hipMemcpyDeviceToHost,
                           q->ctx->stream));
    GBT_HIP(hipStreamSynchronize(q->ctx->stream));
    return GBT_OK;
}

void free_quantizer(gbt_quantizer *q)
{
    if (!q) return;
    gbt_ctx *c = q->ctx;
    (void)hipStreamSynchronize(c->stream);
    dev_free(c, q->keys, q->keys_bytes);
    dev_free(c, q->feats, q->feats_bytes);
    dev_free(c, q->st, kStWords * sizeof(unsigned long long));
    dev_free(c, q->stage, q->stage_bytes);
    dev_free(c, q->enc, q->enc_bytes);
    dev_free(c, q->bkeys, q->bkeys_bytes);
    if (q->ms) {
        merge_sketch_free(c, q->ms);
        delete q->ms;
    }
    if (q->bounce) (void)hipHostFree(q->bounce);
    if (q->mat) gbt_matrix_free(q->mat);
    delete q;
}

// A merged sketch's CSR batch: the batch's (feature, key) pairs grouped by
// feature (counts, then a scatter), summarised and merged.
gbt_status csr_merge_batch(gbt_quantizer *q)
{
    gbt_ctx *c = q->ctx;
    const int32_t m = q->m;
    unsigned long long stv[kStWords];
    GBT_TRY(read_status(q, stv));
    GBT_CHECK(!stv[kStBadIndex], "CSR column indices must be in [0, n_cols) and strictly ascending");
    const int64_t nk = (int64_t)stv[kStKeys];
    if (nk == 0) return GBT_OK;
    unsigned long long *cnt = nullptr;
    GBT_TRY(dev_alloc(c, (size_t)(m + 1) * 8, (void **)&cnt));
    std::vector<unsigned long long> h(m + 1, 0ull), cur(m);
    gbt_status s = GBT_OK;
    auto run = [&]() -> gbt_status {
        GBT_HIP(hipMemcpyAsync(cnt, h.data(), (m + 1) * 8, hipMemcpyHostToDevice, c->stream));
        k_feat_count<<<grid_for(nk, 256), 256, 0, c->stream>>>(q->feats, nk, cnt);
        GBT_LAUNCHED();
        GBT_HIP(hipMemcpyAsync(h.data(), cnt, m * 8, hipMemcpyDeviceToHost, c->stream));
        GBT_HIP(hipStreamSynchronize(c->stream));
        std::vector<int64_t> sb(m), sl(m);
        int64_t o = 0;
        for (int32_t j = 0; j < m; ++j) {
            sb[j] = o;
            sl[j] = (int64_t)h[j];
            cur[j] = (unsigned long long)o;
            o += (int64_t)h[j];
        }
        GBT_TRY(ensure_buf(c, (void **)&q->bkeys, &q->bkeys_bytes, (size_t)nk * 4));
        GBT_HIP(hipMemcpyAsync(cnt, cur.data(), m * 8, hipMemcpyHostToDevice, c->stream));
        k_feat_scatter<<<grid_for(nk, 256), 256, 0, c->stream>>>(q->feats, q->keys, nk, cnt, q->bkeys);
        GBT_LAUNCHED();
        return merge_sketch_add(c, q->ms, q->bkeys, sb.data(), sl.data());
    };
    s = run();
    (void)hipStreamSynchronize(c->stream);
    dev_free(c, cnt, (size_t)(m + 1) * 8);
    return s;
}

}  // namespace

extern "C" {

gbt_status gbt_quantize_begin(gbt_ctx *c, const gbt_quant_params *p, int32_t n_cols,
                              int64_t n_rows_total, int32_t input_kind, gbt_quantizer **out)
{
    GBT_CHECK(c && p && out, "gbt_quantize_begin: NULL argument");
    *out = nullptr;
    GBT_CHECK(p->max_bin >= 2 && p->max_bin <= 65535, "max_bin %d outside [2, 65535]", p->max_bin);
    GBT_CHECK(n_cols > 0, "n_cols must be positive");
    GBT_CHECK(n_rows_total >= 0, "n_rows must be >= 0");
    GBT_CHECK(input_kind == GBT_INPUT_DENSE_F32 || input_kind == GBT_INPUT_CSR_F32,
              "unknown input kind %d", input_kind);
    {
        // a feature takes up to max_bin bins: they must fit a histogram group
        const int32_t lim = hist_feature_bin_limit(input_kind == GBT_INPUT_CSR_F32);
        if (p->max_bin > lim)
            return set_error(GBT_E_UNSUPPORTED, "max_bin %d: the histograms of a %s page hold at most %d bins "
                             "per feature", p->max_bin, input_kind == GBT_INPUT_CSR_F32 ? "sparse" : "dense", lim);
    }
    GBT_CHECK(p->page_home == GBT_HOME_DEVICE || p->page_home == GBT_HOME_PINNED_HOST ||
                  p->page_home == GBT_HOME_DISK,
              "unknown page_home %d", p->page_home);
    GBT_CHECK(p->page_home != GBT_HOME_DISK || (p->page_dir && p->page_dir[0]), "disk pages need page_dir");
    GBT_CHECK(p->page_rows >= 0 && p->sketch_max_rows >= 0, "negative page/sketch rows");
    GBT_CHECK(p->sketch_summary == 0 || (p->sketch_summary >= 2 && p->sketch_summary <= (1 << 20)),
              "sketch_summary %d outside {0} and [2, 2^20]", p->sketch_summary);
    GBT_TRY(set_device(c));
    auto *q = new gbt_quantizer();
    q->ctx = c;
    q->p = *p;
    if (p->page_home == GBT_HOME_DISK) q->dir = p->page_dir;
    q->p.page_dir = nullptr;  // the caller's string is not kept
    if (q->p.sketch_max_rows == 0) q->p.sketch_max_rows = (int64_t)1 << 24;
    q->m = n_cols;
    q->kind = input_kind;
    q->n_total = n_rows_total;
    q->stride = n_rows_total <= q->p.sketch_max_rows
                    ? 1
                    : (n_rows_total + q->p.sketch_max_rows - 1) / q->p.sketch_max_rows;
    gbt_status s = dev_alloc(c, kStWords * sizeof(unsigned long long), (void **)&q->st);
    if (s == GBT_OK) {
        std::vector<unsigned long long> z(kStWords, 0ull);
        hipError_t e = hipMemcpyAsync(q->st, z.data(), kStWords * 8, hipMemcpyHostToDevice, c->stream);
        if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
        if (e != hipSuccess) s = hip_error(e, "status init", __FILE__, __LINE__);
    }
    if (s == GBT_OK && p->sketch_summary > 0) {
        q->ms = new MergeSketch();
        s = merge_sketch_init(c, q->ms, n_cols, p->sketch_summary);
    } else if (s == GBT_OK && input_kind == GBT_INPUT_DENSE_F32) {
        q->n_sketch = (n_rows_total + q->stride - 1) / q->stride;
        q->keys_bytes = (size_t)q->n_sketch * (size_t)n_cols * 4;
        s = dev_alloc(c, q->keys_bytes, (void **)&q->keys);
        if (s != GBT_OK) q->keys_bytes = 0;
    }
    if (s != GBT_OK) {
        free_quantizer(q);
        return s;
    }
    *out = q;
    return GBT_OK;
}

gbt_status gbt_quantize_sketch_batch(gbt_quantizer *q, const gbt_input *batch)
{
    GBT_CHECK(q, "quantizer is NULL");
    GBT_CHECK(!q->cuts_done, "sketch_batch after finalize_cuts");
    gbt_ctx *c = q->ctx;
    GBT_TRY(set_device(c));
    DevBatch b;
    GBT_TRY(stage_batch(q, batch, &b));
    GBT_CHECK(q->sketched_rows + b.rows <= q->n_total, "more rows than announced (%lld)",
              (long long)q->n_total);
    if (b.rows > 0) {
        if (q->kind == GBT_INPUT_DENSE_F32 && q->ms) {
            // Alg. 3: this batch's sample keys, sorted per feature, summarised
            // and merged into the running summaries
            const int64_t g0 = q->sketched_rows, g1 = g0 + b.rows;
            const int64_t s_lo = (g0 + q->stride - 1) / q->stride, s_hi = (g1 + q->stride - 1) / q->stride;
            const int64_t ns = s_hi - s_lo;
            GBT_TRY(ensure_buf(c, (void **)&q->bkeys, &q->bkeys_bytes, std::max<size_t>((size_t)ns * q->m * 4, 16)));
            k_dense_sketch<<<grid_for(b.rows, 256), 256, 0, c->stream>>>(
                b.values, b.rows, q->m, b.ld, g0, q->stride, ns, s_lo, q->bkeys, q->st);
            GBT_LAUNCHED();
            std::vector<int64_t> sb(q->m), sl(q->m, ns);
            for (int32_t j = 0; j < q->m; ++j) sb[j] = (int64_t)j * ns;
            if (ns > 0) GBT_TRY(merge_sketch_add(c, q->ms, q->bkeys, sb.data(), sl.data()));
        } else if (q->kind == GBT_INPUT_DENSE_F32) {
            k_dense_sketch<<<grid_for(b.rows, 256), 256, 0, c->stream>>>(
                b.values, b.rows, q->m, b.ld, q->sketched_rows, q->stride, q->n_sketch, 0, q->keys, q->st);
            GBT_LAUNCHED();
        } else {
            // grow the pair buffers to hold every entry of this batch (a
            // merged sketch keeps one batch's pairs at a time)
            unsigned long long stv[kStWords];
            GBT_TRY(read_status(q, stv));
            if (q->ms && stv[kStKeys]) {
                const unsigned long long zero = 0;
                GBT_HIP(hipMemcpyAsync(q->st + kStKeys, &zero, 8, hipMemcpyHostToDevice, c->stream));
                GBT_HIP(hipStreamSynchronize(c->stream));
                stv[kStKeys] = 0;
            }
            int64_t need = (int64_t)stv[kStKeys] + b.nnz;
            if (need > q->keys_cap) {
                int64_t cap = std::max<int64_t>(need, q->keys_cap * 2);
                uint32_t *nk = nullptr;
                int32_t *nf = nullptr;
                GBT_TRY(dev_alloc(c, (size_t)cap * 4, (void **)&nk));
                gbt_status s = dev_alloc(c, (size_t)cap * 4, (void **)&nf);
                if (s != GBT_OK) {
                    dev_free(c, nk, (size_t)cap * 4);
                    return s;
                }
                if (stv[kStKeys]) {
                    GBT_HIP(hipMemcpyAsync(nk, q->keys, stv[kStKeys] * 4, hipMemcpyDeviceToDevice, c->stream));
                    GBT_HIP(hipMemcpyAsync(nf, q->feats, stv[kStKeys] * 4, hipMemcpyDeviceToDevice, c->stream));
                }
                GBT_HIP(hipStreamSynchronize(c->stream));
                dev_free(c, q->keys, q->keys_bytes);
                dev_free(c, q->feats, q->feats_bytes);
                q->keys = nk;
                q->feats = nf;
                q->keys_bytes = q->feats_bytes = (size_t)cap * 4;
                q->keys_cap = cap;
            }
            k_csr_sketch<<<grid_for(b.rows, 256), 256, 0, c->stream>>>(
                b.indptr, b.indices, b.values, b.rows, q->m, q->sketched_rows, q->stride, q->keys,
                q->feats, q->st);
            GBT_LAUNCHED();
            if (q->ms) GBT_TRY(csr_merge_batch(q));
        }
    }
    q->sketched_rows += b.rows;
    unsigned long long stv[kStWords];
    GBT_TRY(read_status(q, stv));
    GBT_CHECK(!stv[kStInf], "input holds an infinite value");
    GBT_CHECK(!stv[kStBadIndex], "CSR column indices must be in [0, n_cols) and strictly ascending");
    return GBT_OK;
}

static gbt_status finish_cuts(gbt_quantizer *q, std::vector<int32_t> cut_ptr_h, std::vector<float> cut_values_h,
                              std::vector<int64_t> feat_count, const unsigned long long *stv);

// Cuts of a merged sketch from its running summaries: candidate k is the
// value of the first entry whose count reaches ceil(kN/B), duplicates and
// values >= the maximum dropped.
static gbt_status finalize_merged(gbt_quantizer *q, const unsigned long long *stv)
{
    const int32_t m = q->m, B = q->p.max_bin, S = q->ms->S;
    std::vector<uint32_t> v;
    std::vector<long long> cnt;
    std::vector<int64_t> k;
    GBT_TRY(merge_sketch_download(q->ctx, q->ms, &v, &cnt, &k));
    std::vector<int32_t> cut_ptr_h(m + 1, 0);
    std::vector<float> cut_values_h;
    std::vector<int64_t> feat_count;
    for (int32_t j = 0; j < m; ++j) {
        const uint32_t *vj = v.data() + (size_t)j * S;
        const long long *cj = cnt.data() + (size_t)j * S;
        const int64_t kj = k[j];
        const long long N = kj ? cj[kj - 1] : 0;
        feat_count.push_back((int64_t)N);
        if (kj > 0) {
            const uint32_t top = vj[kj - 1];
            int64_t i = 0;
            for (int64_t b = 1; b < B; ++b) {
                const long long target = (b * N + B - 1) / B;
                while (cj[i] < target) ++i;
                if (vj[i] >= top) continue;
                const float x = key_float(vj[i]);
                if (cut_values_h.size() > (size_t)cut_ptr_h[j] && x == cut_values_h.back()) continue;
                cut_values_h.push_back(x);
            }
        }
        cut_ptr_h[j + 1] = (int32_t)cut_values_h.size();
    }
    if (q->kind != GBT_INPUT_CSR_F32) feat_count.clear();
    return finish_cuts(q, std::move(cut_ptr_h), std::move(cut_values_h), std::move(feat_count), stv);
}

gbt_status gbt_quantize_finalize_cuts(gbt_quantizer *q)
{
    GBT_CHECK(q, "quantizer is NULL");
    GBT_CHECK(!q->cuts_done, "finalize_cuts called twice");
    GBT_CHECK(q->sketched_rows == q->n_total, "sketched %lld of %lld rows",
              (long long)q->sketched_rows, (long long)q->n_total);
    gbt_ctx *c = q->ctx;
    GBT_TRY(set_device(c));
    const int32_t m = q->m, B = q->p.max_bin;
    unsigned long long stv[kStWords];
    GBT_TRY(read_status(q, stv));
    if (q->ms) {
        GBT_CHECK(!stv[kStInf], "input holds an infinite value");
        return finalize_merged(q, stv);
    }

    // per-feature key segments
    std::vector<int64_t> seg(m + 1, 0);
    std::vector<int64_t> feat_count;  // CSR: present values per feature in the sketch rows
    uint32_t *keys = q->keys;
    uint32_t *sorted = nullptr;
    size_t sorted_bytes = 0;
    if (q->kind == GBT_INPUT_DENSE_F32) {
        for (int32_t j = 0; j <= m; ++j) seg[j] = (int64_t)j * q->n_sketch;
    } else {
        int64_t nk = (int64_t)stv[kStKeys];
        unsigned long long *cnt = nullptr;
        GBT_TRY(dev_alloc(c, (size_t)(m + 1) * 8, (void **)&cnt));
        std::vector<unsigned long long> h(m + 1, 0ull);
        GBT_HIP(hipMemcpyAsync(cnt, h.data(), (m + 1) * 8, hipMemcpyHostToDevice, c->stream));
        if (nk) {
            k_feat_count<<<grid_for(nk, 256), 256, 0, c->stream>>>(q->feats, nk, cnt);
            GBT_LAUNCHED();
        }
        GBT_HIP(hipMemcpyAsync(h.data(), cnt, m * 8, hipMemcpyDeviceToHost, c->stream));
        GBT_HIP(hipStreamSynchronize(c->stream));
        for (int32_t j = 0; j < m; ++j) seg[j + 1] = seg[j] + (int64_t)h[j];
        feat_count.assign(h.begin(), h.begin() + m);
        std::vector<unsigned long long> cur(m);
        for (int32_t j = 0; j < m; ++j) cur[j] = (unsigned long long)seg[j];
        GBT_HIP(hipMemcpyAsync(cnt, cur.data(), m * 8, hipMemcpyHostToDevice, c->stream));
        sorted_bytes = (size_t)std::max<int64_t>(nk, 1) * 4;
        gbt_status s = dev_alloc(c, sorted_bytes, (void **)&sorted);
        if (s != GBT_OK) {
            dev_free(c, cnt, (size_t)(m + 1) * 8);
            return s;
        }
        if (nk) {
            k_feat_scatter<<<grid_for(nk, 256), 256, 0, c->stream>>>(q->feats, q->keys, nk, cnt, sorted);
            GBT_LAUNCHED();
        }
        GBT_HIP(hipStreamSynchronize(c->stream));
        dev_free(c, cnt, (size_t)(m + 1) * 8);
        keys = sorted;
    }

    // work items: chunks of each feature's segment
    const int64_t kChunk = 1 << 16;
    std::vector<CountWork> work;
    for (int32_t j = 0; j < m; ++j)
        for (int64_t b = seg[j]; b < seg[j + 1]; b += kChunk)
            work.push_back({b, std::min(seg[j + 1], b + kChunk), j, 0});

    // targets per feature: ranks ceil(kN/B)-1 (k=1..B-1) and N-1 (the maximum)
    std::vector<int64_t> N(m, 0);
    std::vector<std::vector<int64_t>> rank(m);
    std::vector<std::vector<uint32_t>> lo(m), hi(m);

    CountWork *work_d = nullptr;
    uint32_t *bounds_d = nullptr;
    int32_t *boff_d = nullptr;
    unsigned int *cnt_d = nullptr;
    size_t work_bytes = std::max<size_t>(work.size(), 1) * sizeof(CountWork);
    size_t bcap = 0;
    gbt_status status = dev_alloc(c, work_bytes, (void **)&work_d);
    if (status == GBT_OK) status = dev_alloc(c, (size_t)(m + 1) * 4, (void **)&boff_d);
    auto cleanup = [&]() {
        (void)hipStreamSynchronize(c->stream);
        dev_free(c, work_d, work_bytes);
        dev_free(c, boff_d, (size_t)(m + 1) * 4);
        dev_free(c, bounds_d, bcap * 4);
        dev_free(c, cnt_d, bcap * 4);
        dev_free(c, sorted, sorted_bytes);
    };
    if (status != GBT_OK) {
        cleanup();
        return status;
    }
    if (!work.empty()) {
        hipError_t e = hipMemcpyAsync(work_d, work.data(), work.size() * sizeof(CountWork),
                                      hipMemcpyHostToDevice, c->stream);
        if (e != hipSuccess) {
            cleanup();
            return hip_error(e, "work upload", __FILE__, __LINE__);
        }
    }

    // One counting pass for the given split points (per feature, sorted and
    // distinct); returns counts per split point.
    auto count_pass = [&](const std::vector<std::vector<uint32_t>> &bnd,
                          std::vector<std::vector<uint32_t>> *out) -> gbt_status {
        std::vector<int32_t> boff(m + 1, 0);
        int32_t maxnb = 0;
        for (int32_t j = 0; j < m; ++j) {
            boff[j + 1] = boff[j] + (int32_t)bnd[j].size();
            maxnb = std::max(maxnb, (int32_t)bnd[j].size());
        }
        size_t total = std::max<size_t>(boff[m], 1);
        if (total > bcap) {
            GBT_HIP(hipStreamSynchronize(c->stream));
            dev_free(c, bounds_d, bcap * 4);
            dev_free(c, cnt_d, bcap * 4);
            bounds_d = nullptr;
            cnt_d = nullptr;
            bcap = 0;
            GBT_TRY(dev_alloc(c, total * 4, (void **)&bounds_d));
            GBT_TRY(dev_alloc(c, total * 4, (void **)&cnt_d));
            bcap = total;
        }
        std::vector<uint32_t> flat;
        flat.reserve(total);
        for (int32_t j = 0; j < m; ++j) flat.insert(flat.end(), bnd[j].begin(), bnd[j].end());
        std::vector<unsigned int> zero(total, 0u);
        if (!flat.empty())
            GBT_HIP(hipMemcpyAsync(bounds_d, flat.data(), flat.size() * 4, hipMemcpyHostToDevice, c->stream));
        GBT_HIP(hipMemcpyAsync(cnt_d, zero.data(), total * 4, hipMemcpyHostToDevice, c->stream));
        GBT_HIP(hipMemcpyAsync(boff_d, boff.data(), (m + 1) * 4, hipMemcpyHostToDevice, c->stream));
        if (!work.empty() && boff[m] > 0) {
            if (maxnb <= kLdsBounds)
                k_bisect_count<true><<<(unsigned)work.size(), 256, 0, c->stream>>>(keys, work_d, bounds_d, boff_d, cnt_d);
            else
                k_bisect_count<false><<<(unsigned)work.size(), 256, 0, c->stream>>>(keys, work_d, bounds_d, boff_d, cnt_d);
            GBT_LAUNCHED();
        }
        std::vector<unsigned int> h(total);
        GBT_HIP(hipMemcpyAsync(h.data(), cnt_d, total * 4, hipMemcpyDeviceToHost, c->stream));
        GBT_HIP(hipStreamSynchronize(c->stream));
        out->assign(m, {});
        for (int32_t j = 0; j < m; ++j) {
            (*out)[j].resize(bnd[j].size());
            uint32_t run = 0;
            for (size_t t = 0; t < bnd[j].size(); ++t) {
                run += h[boff[j] + t];
                (*out)[j][t] = run;  // #keys <= bnd[j][t]
            }
        }
        return GBT_OK;
    };

    // pass 0: N_j = #keys <= largest finite key
    {
        std::vector<std::vector<uint32_t>> bnd(m, std::vector<uint32_t>{kMaxKey}), cnt;
        status = count_pass(bnd, &cnt);
        if (status != GBT_OK) {
            cleanup();
            return status;
        }
        for (int32_t j = 0; j < m; ++j) {
            N[j] = cnt[j][0];
            if (N[j] == 0) continue;
            for (int64_t k = 1; k < B; ++k) rank[j].push_back((k * N[j] + B - 1) / B - 1);
            rank[j].push_back(N[j] - 1);
            lo[j].assign(rank[j].size(), 0u);
            hi[j].assign(rank[j].size(), kMaxKey);
        }
    }
    // bisection passes: the answer for rank r is the least v with #{k <= v} > r
    for (int pass = 0; pass < 16; ++pass) {
        std::vector<std::vector<uint32_t>> bnd(m), cnt;
        bool any = false;
        for (int32_t j = 0; j < m; ++j) {
            auto &b = bnd[j];
            for (size_t t = 0; t < rank[j].size(); ++t) {
                uint64_t l = lo[j][t], h = hi[j][t];
                if (l == h) continue;
                uint64_t len = h - l + 1;
                for (int s = 1; s < kBisectWays; ++s) {
                    uint64_t v = l + (len * (uint64_t)s) / kBisectWays;
                    if (v == 0) continue;
                    v -= 1;  // split point: keys <= v vs > v
                    if (v >= l && v < h) b.push_back((uint32_t)v);
                }
                any = true;
            }
            std::sort(b.begin(), b.end());
            b.erase(std::unique(b.begin(), b.end()), b.end());
        }
        if (!any) break;
        status = count_pass(bnd, &cnt);
        if (status != GBT_OK) {
            cleanup();
            return status;
        }
        for (int32_t j = 0; j < m; ++j) {
            const auto &b = bnd[j];
            for (size_t t = 0; t < rank[j].size(); ++t) {
                uint32_t &l = lo[j][t], &h = hi[j][t];
                if (l == h) continue;
                // narrow [l, h] with every split point inside it
                auto it = std::lower_bound(b.begin(), b.end(), l);
                for (; it != b.end() && *it < h; ++it) {
                    uint32_t c_le = cnt[j][it - b.begin()];
                    if ((int64_t)c_le > rank[j][t]) {
                        h = *it;
                        break;
                    }
                    l = *it + 1;
                }
            }
        }
    }
    cleanup();

    // cuts: distinct candidates strictly below the maximum
    std::vector<int32_t> cut_ptr_h(m + 1, 0);
    std::vector<float> cut_values_h;
    for (int32_t j = 0; j < m; ++j) {
        if (N[j] > 0) {
            GBT_CHECK(lo[j].back() == hi[j].back(), "cut search did not converge");
            float top = key_float(lo[j].back());
            for (size_t t = 0; t + 1 < rank[j].size(); ++t) {
                float v = key_float(lo[j][t]);
                if (v >= top) continue;
                if (cut_values_h.size() > (size_t)cut_ptr_h[j] && v == cut_values_h.back()) continue;
                cut_values_h.push_back(v);
            }
        }
        cut_ptr_h[j + 1] = (int32_t)cut_values_h.size();
    }
    return finish_cuts(q, std::move(cut_ptr_h), std::move(cut_values_h), std::move(feat_count), stv);
}

// The matrix geometry from the cuts (the tail of finalize_cuts for both
// sketches), the cuts on the device, and the sketch state released.
static gbt_status finish_cuts(gbt_quantizer *q, std::vector<int32_t> cut_ptr_h, std::vector<float> cut_values_h,
                              std::vector<int64_t> feat_count, const unsigned long long *stv)
{
    gbt_ctx *c = q->ctx;
    const int32_t m = q->m;
    gbt_matrix *mx = new gbt_matrix();
    q->mat = mx;
    mx->ctx = c;
    mx->feat_count_h = std::move(feat_count);
    mx->n_rows = q->n_total;
    mx->m = m;
    mx->sparse = q->kind == GBT_INPUT_CSR_F32;
    mx->page_home = q->p.page_home;
    mx->page_rows = q->p.page_rows > 0 ? q->p.page_rows : std::max<int64_t>(q->n_total, 1);
    mx->cut_ptr_h = std::move(cut_ptr_h);
    mx->cut_values_h = std::move(cut_values_h);
    mx->bin_ptr_h.assign(m + 1, 0);
    int32_t maxb = 1;
    for (int32_t j = 0; j < m; ++j) {
        int32_t bj = mx->cut_ptr_h[j + 1] - mx->cut_ptr_h[j] + 1;
        maxb = std::max(maxb, bj);
        mx->bin_ptr_h[j + 1] = mx->bin_ptr_h[j] + bj;
    }
    mx->total_bins = mx->bin_ptr_h[m];
    mx->has_missing = stv[kStNan] ? 1 : 0;
    if (mx->sparse) {
        mx->w = std::max(1, ceil_log2_u64((uint64_t)mx->total_bins + 1));
        mx->stride = (int32_t)stv[kStMaxNnz];
        mx->null_sym = (uint32_t)mx->total_bins;
    } else {
        mx->w = std::max(1, ceil_log2_u64((uint64_t)maxb + (mx->has_missing ? 1 : 0)));
        mx->stride = m;
        mx->null_sym = mx->w >= 32 ? 0xffffffffu : ((1u << mx->w) - 1u);
    }
    GBT_CHECK(mx->w <= 32, "symbol width %d exceeds 32 bits", mx->w);
    int64_t words = ((int64_t)mx->stride * mx->w + 31) / 32;
    mx->row_words = (int32_t)std::max<int64_t>(4, (words + 3) / 4 * 4);
    size_t ncut = std::max<size_t>(mx->cut_values_h.size(), 1);
    GBT_TRY(dev_alloc(c, (size_t)(m + 1) * 4, (void **)&mx->cut_ptr_d));
    GBT_TRY(dev_alloc(c, ncut * 4, (void **)&mx->cut_values_d));
    GBT_TRY(dev_alloc(c, (size_t)(m + 1) * 4, (void **)&mx->bin_ptr_d));
    GBT_HIP(hipMemcpyAsync(mx->cut_ptr_d, mx->cut_ptr_h.data(), (m + 1) * 4, hipMemcpyHostToDevice, c->stream));
    if (!mx->cut_values_h.empty())
        GBT_HIP(hipMemcpyAsync(mx->cut_values_d, mx->cut_values_h.data(), mx->cut_values_h.size() * 4,
                               hipMemcpyHostToDevice, c->stream));
    GBT_HIP(hipMemcpyAsync(mx->bin_ptr_d, mx->bin_ptr_h.data(), (m + 1) * 4, hipMemcpyHostToDevice, c->stream));
    GBT_HIP(hipStreamSynchronize(c->stream));
    // the sketch keys are no longer needed
    dev_free(c, q->keys, q->keys_bytes);
    dev_free(c, q->feats, q->feats_bytes);
    q->keys = nullptr;
    q->feats = nullptr;
    q->keys_bytes = q->feats_bytes = 0;
    dev_free(c, q->bkeys, q->bkeys_bytes);
    q->bkeys = nullptr;
    q->bkeys_bytes = 0;
    if (q->ms) {
        merge_sketch_free(c, q->ms);
        delete q->ms;
        q->ms = nullptr;
    }
    q->cuts_done = true;
    return GBT_OK;
}

gbt_status gbt_quantize_encode_batch(gbt_quantizer *q, const gbt_input *batch)
{
    GBT_CHECK(q, "quantizer is NULL");
    GBT_CHECK(q->cuts_done, "encode_batch before finalize_cuts");
    gbt_ctx *c = q->ctx;
    gbt_matrix *mx = q->mat;
    GBT_TRY(set_device(c));
    DevBatch b;
    GBT_TRY(stage_batch(q, batch, &b));
    GBT_CHECK(q->encoded_rows + b.rows <= q->n_total, "more rows than announced");
    if (b.rows == 0) return GBT_OK;
    size_t bytes = (size_t)b.rows * mx->row_words * 4;
    GBT_TRY(ensure_buf(c, (void **)&q->enc, &q->enc_bytes, bytes));
    if (!mx->sparse)
        k_encode_dense<<<grid_for(b.rows, 256), 256, 0, c->stream>>>(
            b.values, b.rows, mx->m, b.ld, mx->cut_ptr_d, mx->cut_values_d, mx->w, mx->row_words,
            mx->null_sym, q->enc);
    else
        k_encode_csr<<<grid_for(b.rows, 256), 256, 0, c->stream>>>(
            b.indptr, b.indices, b.values, b.rows, mx->cut_ptr_d, mx->cut_values_d, mx->bin_ptr_d,
            mx->w, mx->stride, mx->row_words, mx->null_sym, q->enc, q->st);
    GBT_LAUNCHED();
    // copy the encoded rows into their pages
    int64_t r = q->encoded_rows, end = r + b.rows;
    while (r < end) {
        int64_t pi = r / mx->page_rows;
        int64_t p0 = pi * mx->page_rows, prow = std::min(mx->page_rows, mx->n_rows - p0);
        while ((int64_t)mx->pages.size() <= pi) {
            GbtPage pg;
            pg.row0 = (int64_t)mx->pages.size() * mx->page_rows;
            pg.rows = std::min(mx->page_rows, mx->n_rows - pg.row0);
            size_t pb = (size_t)std::max<int64_t>(pg.rows, 1) * mx->row_words * 4;
            if (mx->page_home == GBT_HOME_PINNED_HOST) {
                pg.host = true;
                // mapped: the gather compaction reads kept rows in place
                hipError_t e = hipHostMalloc((void **)&pg.words, pb, hipHostMallocMapped);
                if (e != hipSuccess) {
                    (void)hipGetLastError();
                    return set_error(GBT_E_OOM, "hipHostMalloc(%zu) for a page failed", pb);
                }
            } else if (mx->page_home == GBT_HOME_DISK) {
                char name[64];
                snprintf(name, sizeof name, "/gbt-%d-%llu-%zu.pages", (int)getpid(),
                         (unsigned long long)mx->uid, mx->pages.size());
                const std::string path = q->dir + name;
                pg.fd = open(path.c_str(), O_RDWR | O_CREAT | O_EXCL | O_CLOEXEC, 0600);
                if (pg.fd < 0) return set_error(GBT_E_IO, "cannot create %s: %s", path.c_str(), strerror(errno));
                (void)unlink(path.c_str());  // the open descriptor keeps the file
                mx->pages.push_back(pg);
                continue;
            } else {
                GBT_TRY(dev_alloc(c, pb, (void **)&pg.words));
            }
            mx->pages.push_back(pg);
        }
        int64_t take = std::min(end, p0 + prow) - r;
        GbtPage &pg = mx->pages[pi];
        if (pg.fd >= 0) {
            const size_t bytes = (size_t)take * mx->row_words * 4;
            if (q->bounce_bytes < bytes) {
                GBT_HIP(hipStreamSynchronize(c->stream));
                if (q->bounce) GBT_HIP(hipHostFree(q->bounce));
                q->bounce = nullptr;
                q->bounce_bytes = 0;
                GBT_HIP(hipHostMalloc(&q->bounce, bytes, hipHostMallocDefault));
                q->bounce_bytes = bytes;
            }
            GBT_HIP(hipMemcpyAsync(q->bounce, q->enc + (r - q->encoded_rows) * mx->row_words, bytes,
                                   hipMemcpyDeviceToHost, c->stream));
            GBT_HIP(hipStreamSynchronize(c->stream));
            GBT_TRY(file_write(pg.fd, q->bounce, bytes, (r - p0) * mx->row_words * 4));
            r += take;
            continue;
        }
        GBT_HIP(hipMemcpyAsync(pg.words + (r - p0) * mx->row_words,
                               q->enc + (r - q->encoded_rows) * mx->row_words,
                               (size_t)take * mx->row_words * 4,
                               pg.host ? hipMemcpyDeviceToHost : hipMemcpyDeviceToDevice, c->stream));
        r += take;
    }
    q->encoded_rows = end;
    unsigned long long stv[kStWords];
    GBT_TRY(read_status(q, stv));
    GBT_CHECK(!stv[kStBadIndex], "encode batch differs from the sketched batches");
    return GBT_OK;
}

gbt_status gbt_quantize_end(gbt_quantizer *q, gbt_matrix **out)
{
    GBT_CHECK(q && out, "gbt_quantize_end: NULL argument");
    *out = nullptr;
    GBT_CHECK(q->cuts_done && q->encoded_rows == q->n_total, "encoded %lld of %lld rows",
              (long long)q->encoded_rows, (long long)q->n_total);
    if (q->mat->pages.empty()) {  // zero rows: one empty page keeps the geometry usable
        GbtPage pg;
        GBT_TRY(dev_alloc(q->ctx, (size_t)q->mat->row_words * 4, (void **)&pg.words));
        q->mat->pages.push_back(pg);
    }
    *out = q->mat;
    q->mat = nullptr;
    free_quantizer(q);
    return GBT_OK;
}

gbt_status gbt_quantizer_free(gbt_quantizer *q)
{
    free_quantizer(q);
    return GBT_OK;
}

gbt_status gbt_quantize(gbt_ctx *c, const gbt_input *in, const gbt_quant_params *p,
                        gbt_matrix **out)
{
    GBT_CHECK(c && in && p && out, "gbt_quantize: NULL argument");
    *out = nullptr;
    gbt_quantizer *q = nullptr;
    GBT_TRY(gbt_quantize_begin(c, p, in->n_cols, in->n_rows, in->kind, &q));
    gbt_status s = gbt_quantize_sketch_batch(q, in);
    if (s == GBT_OK) s = gbt_quantize_finalize_cuts(q);
    if (s == GBT_OK) s = gbt_quantize_encode_batch(q, in);
    if (s != GBT_OK) {
        free_quantizer(q);
        return s;
    }
    return gbt_quantize_end(q, out);
}

gbt_status gbt_matrix_info_get(const gbt_matrix *mx, gbt_matrix_info *info)
{
    GBT_CHECK(mx && info, "gbt_matrix_info_get: NULL argument");
    info->n_rows = mx->n_rows;
    info->n_cols = mx->m;
    info->sparse = mx->sparse;
    info->has_missing = mx->has_missing;
    info->symbol_bits = mx->w;
    info->stride = mx->stride;
    info->row_words = mx->row_words;
    info->null_symbol = mx->null_sym;
    info->n_pages = (int32_t)mx->pages.size();
    info->total_bins = mx->total_bins;
    info->page_rows = mx->page_rows;
    info->page_home = mx->page_home;
    info->pad0 = 0;
    return GBT_OK;
}

gbt_status gbt_matrix_get_cuts(const gbt_matrix *mx, int32_t *cut_ptr_h, float *cut_values_h)
{
    GBT_CHECK(mx, "matrix is NULL");
    if (cut_ptr_h) memcpy(cut_ptr_h, mx->cut_ptr_h.data(), (mx->m + 1) * 4);
    if (cut_values_h && !mx->cut_values_h.empty())
        memcpy(cut_values_h, mx->cut_values_h.data(), mx->cut_values_h.size() * 4);
    return GBT_OK;
}

gbt_status gbt_matrix_page_rows(const gbt_matrix *mx, int32_t page, int64_t *row0, int64_t *rows)
{
    GBT_CHECK(mx && page >= 0 && page < (int32_t)mx->pages.size(), "bad page index %d", page);
    if (row0) *row0 = mx->pages[page].row0;
    if (rows) *rows = mx->pages[page].rows;
    return GBT_OK;
}

gbt_status gbt_matrix_copy_page(const gbt_matrix *mx, int32_t page, void *dst, int64_t dst_words)
{
    GBT_CHECK(mx && dst && page >= 0 && page < (int32_t)mx->pages.size(), "bad page copy request");
    const GbtPage &pg = mx->pages[page];
    int64_t words = pg.rows * mx->row_words;
    GBT_CHECK(dst_words >= words, "destination holds %lld words, page has %lld",
              (long long)dst_words, (long long)words);
    GBT_TRY(set_device(mx->ctx));
    GBT_HIP(hipStreamSynchronize(mx->ctx->stream));
    if (words && pg.fd >= 0) {
        std::vector<uint32_t> tmp((size_t)words);
        GBT_TRY(file_read(pg.fd, tmp.data(), (size_t)words * 4, 0));
        GBT_HIP(hipMemcpy(dst, tmp.data(), (size_t)words * 4, hipMemcpyDefault));
    } else if (words) {
        GBT_HIP(hipMemcpy(dst, pg.words, (size_t)words * 4, hipMemcpyDefault));
    }
    return GBT_OK;
}

gbt_status gbt_matrix_free(gbt_matrix *mx)
{
    if (!mx) return GBT_OK;
    gbt_ctx *c = mx->ctx;
    (void)hipSetDevice(c->device);
    (void)hipStreamSynchronize(c->stream);
    (void)hipStreamSynchronize(c->side);
    for (auto &pg : mx->pages) {
        if (pg.fd >= 0)
            (void)close(pg.fd);
        else if (pg.host)
            (void)hipHostFree(pg.words);
        else
            dev_free(c, pg.words, (size_t)std::max<int64_t>(pg.rows, 1) * mx->row_words * 4);
    }
    dev_free(c, mx->cut_ptr_d, (size_t)(mx->m + 1) * 4);
    dev_free(c, mx->cut_values_d, std::max<size_t>(mx->cut_values_h.size(), 1) * 4);
    dev_free(c, mx->bin_ptr_d, (size_t)(mx->m + 1) * 4);
    if (mx->groups_d) dev_free(c, mx->groups_d, mx->groups_bytes);
    delete mx;
    return GBT_OK;
}

}  // extern "C"
