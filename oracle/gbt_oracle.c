/*
 * gbt_oracle.c -- CPU oracle for one boosting iteration of out-of-core GPU
 * gradient boosting (Ou, "Out-of-Core GPU Gradient Boosting", KDD 2020).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, plain, obviously correct
 * definition that the HIP path is checked against.  Only the tests, the smoke
 * check and the benchmark's CPU-baseline leg may load it.  It shares no code,
 * header, table or constant generator with the HIP library: every rule below
 * is written out again from the paper and from the readings recorded in the
 * design notes.
 *
 * Built with -O2 -ffp-contract=off and no fast-math, so every floating-point
 * operation is the single IEEE operation written here.  The plain build is
 * single threaded.  A second build with -fopenmp spreads the loops marked
 * "omp" over threads; each such loop either treats rows (or features)
 * independently or reduces integers or maxima, whose results do not depend
 * on the order, so both builds return the same bits (a CPU test checks
 * whole trees).
 *
 * Contents, in the order the paper presents them:
 *   orc_exp / orc_philox4x64_10 ...... helpers (Cody-Waite exp; Philox of
 *                                       Salmon et al., SC'11)
 *   orc_sketch_cuts_* ................ Sec. 3.1 (Alg. 2/3): quantile cuts,
 *                                       exact and batch-merged (Alg. 3)
 *   orc_bin_* / orc_ellpack_* ........ Sec. 2.2 + Sec. 3.2 (Alg. 4/5): bins
 *                                       and bit-packed ELLPACK rows
 *   orc_gradients .................... Sec. 2.1, Eq. 4-5: g and h
 *   orc_mvs_* ........................ Sec. 2.4 Eq. 9 + Sec. 3.4 (Alg. 7):
 *                                       minimal variance sampling
 *   orc_sgb_* / orc_goss_* ........... Sec. 2.3: the SGB and GOSS samplers
 *   orc_fixed_point .................. exact integer gradient sums
 *   orc_build_hist ................... Alg. 1 BuildHistograms
 *   orc_eval_node .................... Alg. 1 EvaluateSplit with Eq. 8
 *   orc_partition .................... Alg. 1 RepartitionInstances
 *   orc_leaf_value ................... Eq. 6
 *   orc_train_tree ................... Alg. 7 then Alg. 1, level by level
 *   orc_predict_* .................... Eq. 1
 *
 * Parity status: every function here is pinned by a CPU test against
 * something other than itself (closed forms, brute force, numpy/sklearn
 * routines, invariants); see the tests named test_oracle_*.py.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORC_OK 0
#define ORC_EINVAL (-1)
#define ORC_ENOMEM (-2)

#define ORC_MISSING 0xFFFFu

#define ORC_LOSS_LOGISTIC 0
#define ORC_LOSS_SQUARED 1

#define ORC_NODE_PRESENT 1u
#define ORC_NODE_LEAF 2u
#define ORC_NODE_DEFAULT_LEFT 4u

/* Threads of the omp build (n > 0 sets them); 1 for the plain build. */
int32_t orc_threads(int32_t n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
    return (int32_t)omp_get_max_threads();
#else
    (void)n;
    return 1;
#endif
}

/* ------------------------------------------------------------------------ */
/* Data types shared with oracle.py (ctypes mirrors them field by field).    */
/* ------------------------------------------------------------------------ */

/* A binned matrix: either dense bins (n x m, ORC_MISSING for a missing
 * value) or CSR bins (only the present entries, features ascending within
 * a row). */
typedef struct {
    int64_t n;
    int32_t m;
    int32_t pad0;
    const uint16_t *dense;   /* n*m or NULL */
    const int64_t *indptr;   /* n+1 (CSR) */
    const int32_t *feat;     /* nnz (CSR) */
    const uint16_t *bin;     /* nnz (CSR) */
    const int32_t *nbins;    /* B_j, m entries */
    const int32_t *cut_ptr;  /* m+1 */
    const float *cut_values; /* cut_ptr[m] */
} orc_data;

typedef struct {
    int32_t loss;
    int32_t max_depth;
    double eta;
    double lambda;
    double gamma;
    double min_child_weight;
    double f;          /* sampling fraction; 1 means no sampling */
    double mvs_lambda; /* the lambda of Eq. 9 */
    uint64_t seed;
    uint64_t iteration;
    int32_t sampler;   /* ORC_SAMPLE_MVS, _SGB or _GOSS (used when f < 1) */
    int32_t pad0;
    double goss_a;     /* GOSS: the top fraction a (the rest fraction is f - a) */
} orc_params;

enum { ORC_SAMPLE_MVS = 0, ORC_SAMPLE_SGB = 1, ORC_SAMPLE_GOSS = 2 };

typedef struct {
    int32_t feature;
    int32_t split_bin;
    float threshold;
    float leaf_value;
    double gain;
    int64_t sum_g;
    int64_t sum_h;
    int32_t n_rows;
    uint8_t flags;
    uint8_t pad[3];
} orc_node;

typedef struct {
    double gain;
    int64_t left_g, left_h, right_g, right_h;
    int32_t feature;
    int32_t split_bin;
    int32_t default_left;
    int32_t valid;
} orc_split;

typedef struct {
    int64_t n_sampled;
    int64_t K;
    int64_t T;
    int32_t e_key;
    int32_t e_g;
    int32_t e_h;
    int32_t n_nodes;
} orc_info;

/* ------------------------------------------------------------------------ */
/* exp(x): Cody & Waite argument reduction (Software Manual for the          */
/* Elementary Functions, 1980) with ln 2 split into a 32-significant-bit      */
/* head and a tail, then the Taylor series of e^r to degree 13 in Horner      */
/* form with explicit fused multiply-adds, then scaling by 2^k.               */
/*   ln2_hi = ln 2 rounded to double with its low 21 significand bits        */
/*            cleared (so k*ln2_hi is exact for |k| < 2^21)                   */
/*   ln2_lo = nearest double to (ln 2 - ln2_hi)                               */
/*   c_k    = nearest double to 1/k!                                          */
/* |r| <= ln2/2 so the truncation term r^14/14! is below 2^-60.  Inputs       */
/* outside [-708, 708] are clamped to 0 or +inf, which keeps every result     */
/* normal; the logistic sigmoid never sees the difference.                    */
/* ------------------------------------------------------------------------ */
double orc_exp(double x)
{
    const double ln2_hi = 0x1.62e42fee00000p-1;
    const double ln2_lo = 0x1.a39ef35793c76p-33;
    const double inv_ln2 = 0x1.71547652b82fep+0;
    if (isnan(x)) return x;
    if (x > 708.0) return INFINITY;
    if (x < -708.0) return 0.0;
    double k = rint(x * inv_ln2);
    double r = (x - k * ln2_hi) - k * ln2_lo;
    double p = 0x1.6124613a86d09p-33;        /* 1/13! */
    p = fma(p, r, 0x1.1eed8eff8d898p-29);    /* 1/12! */
    p = fma(p, r, 0x1.ae64567f544e4p-26);    /* 1/11! */
    p = fma(p, r, 0x1.27e4fb7789f5cp-22);    /* 1/10! */
    p = fma(p, r, 0x1.71de3a556c734p-19);    /* 1/9!  */
    p = fma(p, r, 0x1.a01a01a01a01ap-16);    /* 1/8!  */
    p = fma(p, r, 0x1.a01a01a01a01ap-13);    /* 1/7!  */
    p = fma(p, r, 0x1.6c16c16c16c17p-10);    /* 1/6!  */
    p = fma(p, r, 0x1.1111111111111p-7);     /* 1/5!  */
    p = fma(p, r, 0x1.5555555555555p-5);     /* 1/4!  */
    p = fma(p, r, 0x1.5555555555555p-3);     /* 1/3!  */
    p = fma(p, r, 0.5);                      /* 1/2!  */
    p = fma(p, r, 1.0);
    p = fma(p, r, 1.0);
    return ldexp(p, (int)k);
}

/* ------------------------------------------------------------------------ */
/* Philox4x64-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as   */
/* easy as 1, 2, 3", SC'11).  Ten rounds; the key is bumped by the Weyl      */
/* constants between rounds.                                                 */
/* ------------------------------------------------------------------------ */
void orc_philox4x64_10(const uint64_t ctr[4], const uint64_t key[2], uint64_t out[4])
{
    const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
    const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
    uint64_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
    uint64_t k0 = key[0], k1 = key[1];
    for (int round = 0; round < 10; ++round) {
        if (round > 0) {
            k0 += W0;
            k1 += W1;
        }
        unsigned __int128 p0 = (unsigned __int128)M0 * c0;
        unsigned __int128 p1 = (unsigned __int128)M1 * c2;
        uint64_t hi0 = (uint64_t)(p0 >> 64), lo0 = (uint64_t)p0;
        uint64_t hi1 = (uint64_t)(p1 >> 64), lo1 = (uint64_t)p1;
        uint64_t n0 = hi1 ^ c1 ^ k0;
        uint64_t n2 = hi0 ^ c3 ^ k1;
        c0 = n0;
        c1 = lo1;
        c2 = n2;
        c3 = lo0;
    }
    out[0] = c0;
    out[1] = c1;
    out[2] = c2;
    out[3] = c3;
}

/* ------------------------------------------------------------------------ */
/* Sec. 3.1, Alg. 2/3: quantile cuts.  Quantiles are cut points that split   */
/* a feature's range into intervals of equal probability.  Exact reading:    */
/* sort the sketch values s_0..s_{N-1}; candidate k (1..B-1) is              */
/* s[ceil(k*N/B) - 1]; drop duplicates and any candidate >= s_{N-1}.         */
/* bin(x) = number of cuts strictly below x.                                 */
/* ------------------------------------------------------------------------ */
static int cmp_float(const void *a, const void *b)
{
    float x = *(const float *)a, y = *(const float *)b;
    return (x > y) - (x < y);
}

/* Cuts of one feature from its N sketch values (NaN already removed,
 * -0 already made +0).  Writes at most B-1 cuts; returns their count. */
static int32_t cuts_from_values(float *vals, int64_t N, int32_t B, float *out)
{
    if (N <= 0) return 0;
    qsort(vals, (size_t)N, sizeof(float), cmp_float);
    float top = vals[N - 1];
    int32_t c = 0;
    for (int64_t k = 1; k < B; ++k) {
        int64_t idx = (k * N + B - 1) / B - 1;
        float t = vals[idx];
        if (t >= top) continue;
        if (c > 0 && t == out[c - 1]) continue;
        out[c++] = t;
    }
    return c;
}

static int64_t sketch_stride(int64_t n, int64_t sketch_max_rows)
{
    if (n <= sketch_max_rows) return 1;
    return (n + sketch_max_rows - 1) / sketch_max_rows;
}

/* Dense float input (row-major, leading dimension ld).  cut_values must
 * hold m*(max_bin-1) floats.  Returns ORC_OK or ORC_EINVAL (+-inf seen). */
int orc_sketch_cuts_dense(const float *X, int64_t n, int32_t m, int64_t ld, int32_t max_bin,
                          int64_t sketch_max_rows, int32_t *cut_ptr, float *cut_values)
{
    if (n < 0 || m <= 0 || max_bin < 2 || ld < m) return ORC_EINVAL;
    int64_t stride = sketch_stride(n, sketch_max_rows);
    /* each feature's cuts go to its own max_bin-1 slots first, then are
     * packed in feature order */
    float *tmp = (float *)malloc(sizeof(float) * (size_t)m * (size_t)(max_bin - 1));
    int32_t *cnt = (int32_t *)malloc(sizeof(int32_t) * (size_t)m);
    if (!tmp || !cnt) {
        free(tmp);
        free(cnt);
        return ORC_ENOMEM;
    }
    int bad = 0, oom = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : bad, oom)
    for (int32_t j = 0; j < m; ++j) {
        float *vals = (float *)malloc(sizeof(float) * (size_t)(n / stride + 1));
        cnt[j] = 0;
        if (!vals) {
            oom = 1;
            continue;
        }
        int64_t N = 0;
        for (int64_t i = 0; i < n; i += stride) {
            float x = X[i * ld + j];
            if (isnan(x)) continue;
            if (isinf(x)) {
                bad = 1;
                break;
            }
            if (x == 0.0f) x = 0.0f; /* -0 -> +0 */
            vals[N++] = x;
        }
        cnt[j] = cuts_from_values(vals, N, max_bin, tmp + (size_t)j * (size_t)(max_bin - 1));
        free(vals);
    }
    if (!bad && !oom) {
        cut_ptr[0] = 0;
        for (int32_t j = 0; j < m; ++j) {
            memcpy(cut_values + cut_ptr[j], tmp + (size_t)j * (size_t)(max_bin - 1), sizeof(float) * (size_t)cnt[j]);
            cut_ptr[j + 1] = cut_ptr[j] + cnt[j];
        }
    }
    free(tmp);
    free(cnt);
    return oom ? ORC_ENOMEM : (bad ? ORC_EINVAL : ORC_OK);
}

/* CSR float input: absent entries and NaN values are missing. */
int orc_sketch_cuts_csr(const int64_t *indptr, const int32_t *indices, const float *values,
                        int64_t n, int32_t m, int32_t max_bin, int64_t sketch_max_rows,
                        int32_t *cut_ptr, float *cut_values)
{
    if (n < 0 || m <= 0 || max_bin < 2) return ORC_EINVAL;
    int64_t stride = sketch_stride(n, sketch_max_rows);
    /* gather the sketch entries per feature */
    int64_t *cnt = (int64_t *)calloc((size_t)m + 1, sizeof(int64_t));
    if (!cnt) return ORC_ENOMEM;
    for (int64_t i = 0; i < n; i += stride)
        for (int64_t e = indptr[i]; e < indptr[i + 1]; ++e) {
            float x = values[e];
            if (indices[e] < 0 || indices[e] >= m) {
                free(cnt);
                return ORC_EINVAL;
            }
            if (isinf(x)) {
                free(cnt);
                return ORC_EINVAL;
            }
            if (!isnan(x)) cnt[indices[e] + 1]++;
        }
    for (int32_t j = 0; j < m; ++j) cnt[j + 1] += cnt[j];
    float *vals = (float *)malloc(sizeof(float) * (size_t)(cnt[m] + 1));
    int64_t *fill = (int64_t *)malloc(sizeof(int64_t) * (size_t)m);
    if (!vals || !fill) {
        free(cnt);
        free(vals);
        free(fill);
        return ORC_ENOMEM;
    }
    for (int32_t j = 0; j < m; ++j) fill[j] = cnt[j];
    for (int64_t i = 0; i < n; i += stride)
        for (int64_t e = indptr[i]; e < indptr[i + 1]; ++e) {
            float x = values[e];
            if (isnan(x)) continue;
            if (x == 0.0f) x = 0.0f;
            vals[fill[indices[e]]++] = x;
        }
    float *tmp = (float *)malloc(sizeof(float) * (size_t)m * (size_t)(max_bin - 1));
    int32_t *nc = (int32_t *)malloc(sizeof(int32_t) * (size_t)m);
    if (!tmp || !nc) {
        free(vals);
        free(fill);
        free(cnt);
        free(tmp);
        free(nc);
        return ORC_ENOMEM;
    }
#pragma omp parallel for schedule(dynamic, 1)
    for (int32_t j = 0; j < m; ++j)
        nc[j] = cuts_from_values(vals + cnt[j], cnt[j + 1] - cnt[j], max_bin,
                                 tmp + (size_t)j * (size_t)(max_bin - 1));
    cut_ptr[0] = 0;
    for (int32_t j = 0; j < m; ++j) {
        memcpy(cut_values + cut_ptr[j], tmp + (size_t)j * (size_t)(max_bin - 1), sizeof(float) * (size_t)nc[j]);
        cut_ptr[j + 1] = cut_ptr[j] + nc[j];
    }
    free(tmp);
    free(nc);
    free(vals);
    free(fill);
    free(cnt);
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Sec. 3.1, Alg. 3: the out-of-core sketch.  The sketch sample (the rows    */
/* above) arrives in batches, and each batch's column cuts are folded into   */
/* one running summary per feature.  The paper leaves the folding open;      */
/* reading: a summary is a list of distinct values v_1 < ... < v_k, each     */
/* with an estimate c_i of the number of sample values <= v_i (c_k = N, the  */
/* values summarised).                                                       */
/*   batch summary: the batch's sorted values; all its distinct values with  */
/*     their exact counts, pruned to S entries.                              */
/*   merge(A, B): every value of A or B, with c(v) = c_A(v) + c_B(v), where  */
/*     c_X(v) is the count of X's last entry <= v (0 if none); pruned to S.  */
/*   prune to S (when k > S): for t = 1..S the entry i_t = min{ i : c_i >=   */
/*     ceil(t N / S) }, each entry kept once (i_S = k: the maximum stays).   */
/*   running summary: R_b = merge(R_{b-1}, summary of batch b), batch order. */
/*   cuts: candidate j (1..B-1) is the value of min{ i : c_i >= ceil(jN/B) }; */
/*     duplicates and values >= v_k dropped, as for the exact rule.          */
/* When no summary ever exceeds S entries every count is exact and the cuts  */
/* equal the exact rule's over the whole sample.  Otherwise each prune and   */
/* merge can only lower a count: c(v) <= the true count of values <= v.      */
/* ------------------------------------------------------------------------ */
typedef struct {
    float v;
    int64_t c;
} orc_entry;

/* Prune k entries (in) over N values to at most S (out, separate). */
static int64_t summary_prune(const orc_entry *in, int64_t k, int64_t N, int32_t S, orc_entry *out)
{
    if (k <= S) {
        memcpy(out, in, sizeof(orc_entry) * (size_t)k);
        return k;
    }
    int64_t o = 0, i = 0, last = -1;
    for (int64_t t = 1; t <= S; ++t) {
        int64_t target = (t * N + S - 1) / S;
        while (in[i].c < target) ++i;
        if (i != last) out[o++] = in[i];
        last = i;
    }
    return o;
}

/* The exact summary of n sorted values (distinct values, counts <= each). */
static int64_t summary_of_sorted(const float *vals, int64_t n, orc_entry *out)
{
    int64_t k = 0;
    for (int64_t i = 0; i < n; ++i)
        if (i == n - 1 || vals[i] != vals[i + 1]) {
            out[k].v = vals[i];
            out[k].c = i + 1;
            ++k;
        }
    return k;
}

static int64_t summary_merge(const orc_entry *A, int64_t ka, const orc_entry *B, int64_t kb, orc_entry *U)
{
    int64_t i = 0, j = 0, k = 0, ca = 0, cb = 0;
    while (i < ka || j < kb) {
        float v;
        if (j >= kb || (i < ka && A[i].v < B[j].v)) {
            v = A[i].v;
            ca = A[i].c;
            ++i;
        } else if (i >= ka || B[j].v < A[i].v) {
            v = B[j].v;
            cb = B[j].c;
            ++j;
        } else {
            v = A[i].v;
            ca = A[i].c;
            cb = B[j].c;
            ++i;
            ++j;
        }
        U[k].v = v;
        U[k].c = ca + cb;
        ++k;
    }
    return k;
}

/* The running summary of one feature after one more batch of n values
 * (NaN removed, -0 made +0; vals is sorted in place). */
static int summary_add_batch(orc_entry **R, int64_t *kR, float *vals, int64_t n, int32_t S)
{
    if (n <= 0) return ORC_OK;
    qsort(vals, (size_t)n, sizeof(float), cmp_float);
    orc_entry *e = (orc_entry *)malloc(sizeof(orc_entry) * (size_t)n);
    orc_entry *b = (orc_entry *)malloc(sizeof(orc_entry) * (size_t)(S + 1));
    orc_entry *u = (orc_entry *)malloc(sizeof(orc_entry) * (size_t)(*kR + S + 1));
    orc_entry *r = (orc_entry *)malloc(sizeof(orc_entry) * (size_t)(S + 1));
    if (!e || !b || !u || !r) {
        free(e);
        free(b);
        free(u);
        free(r);
        return ORC_ENOMEM;
    }
    int64_t ke = summary_of_sorted(vals, n, e);
    int64_t kb = summary_prune(e, ke, n, S, b);
    int64_t NR = *kR ? (*R)[*kR - 1].c : 0;
    int64_t ku = summary_merge(*R, *kR, b, kb, u);
    int64_t kr = summary_prune(u, ku, NR + n, S, r);
    free(e);
    free(b);
    free(u);
    free(*R);
    *R = r;
    *kR = kr;
    return ORC_OK;
}

/* Cuts of one feature from its summary (at most B-1; returns their count). */
static int32_t cuts_from_summary(const orc_entry *R, int64_t k, int32_t B, float *out)
{
    if (k <= 0) return 0;
    int64_t N = R[k - 1].c;
    float top = R[k - 1].v;
    int32_t c = 0;
    int64_t i = 0;
    for (int64_t j = 1; j < B; ++j) {
        int64_t target = (j * N + B - 1) / B;
        while (R[i].c < target) ++i;
        float t = R[i].v;
        if (t >= top) continue;
        if (c > 0 && t == out[c - 1]) continue;
        out[c++] = t;
    }
    return c;
}

/* Dense input in batches of batch_rows rows (the last one shorter).  The
 * sketch sample is the rows of the exact rule (stride from n and
 * sketch_max_rows); summary_size = S >= 2.  Same outputs as
 * orc_sketch_cuts_dense; entries_out (optional) receives each feature's
 * final summary size. */
int orc_sketch_cuts_merge_dense(const float *X, int64_t n, int32_t m, int64_t ld, int32_t max_bin,
                                int64_t sketch_max_rows, int32_t S, int64_t batch_rows, int32_t *cut_ptr,
                                float *cut_values, int64_t *entries_out)
{
    if (n < 0 || m <= 0 || max_bin < 2 || ld < m || S < 2 || batch_rows <= 0) return ORC_EINVAL;
    int64_t stride = sketch_stride(n, sketch_max_rows);
    float *tmp = (float *)malloc(sizeof(float) * (size_t)m * (size_t)(max_bin - 1));
    int32_t *cnt = (int32_t *)malloc(sizeof(int32_t) * (size_t)m);
    if (!tmp || !cnt) {
        free(tmp);
        free(cnt);
        return ORC_ENOMEM;
    }
    int bad = 0, oom = 0;
    /* omp: features are independent */
#pragma omp parallel for schedule(dynamic, 1) reduction(| : bad, oom)
    for (int32_t j = 0; j < m; ++j) {
        orc_entry *R = NULL;
        int64_t kR = 0;
        float *vals = (float *)malloc(sizeof(float) * (size_t)(batch_rows / stride + 2));
        cnt[j] = 0;
        if (!vals) {
            oom = 1;
            continue;
        }
        for (int64_t b0 = 0; b0 < n && !bad && !oom; b0 += batch_rows) {
            int64_t b1 = b0 + batch_rows < n ? b0 + batch_rows : n, N = 0;
            for (int64_t i = (b0 + stride - 1) / stride * stride; i < b1; i += stride) {
                float x = X[i * ld + j];
                if (isnan(x)) continue;
                if (isinf(x)) {
                    bad = 1;
                    break;
                }
                if (x == 0.0f) x = 0.0f;
                vals[N++] = x;
            }
            if (!bad && summary_add_batch(&R, &kR, vals, N, S) != ORC_OK) oom = 1;
        }
        if (!bad && !oom) cnt[j] = cuts_from_summary(R, kR, max_bin, tmp + (size_t)j * (size_t)(max_bin - 1));
        if (entries_out) entries_out[j] = kR;
        free(R);
        free(vals);
    }
    if (!bad && !oom) {
        cut_ptr[0] = 0;
        for (int32_t j = 0; j < m; ++j) {
            memcpy(cut_values + cut_ptr[j], tmp + (size_t)j * (size_t)(max_bin - 1), sizeof(float) * (size_t)cnt[j]);
            cut_ptr[j + 1] = cut_ptr[j] + cnt[j];
        }
    }
    free(tmp);
    free(cnt);
    return oom ? ORC_ENOMEM : (bad ? ORC_EINVAL : ORC_OK);
}

/* The final running summary of feature j of dense input (as in
 * orc_sketch_cuts_merge_dense): its k entries (returned) into v[], c[]
 * (room for S entries), or -1 on error. */
int64_t orc_sketch_summary_dense(const float *X, int64_t n, int32_t m, int64_t ld, int64_t sketch_max_rows,
                                 int32_t S, int64_t batch_rows, int32_t j, float *v, int64_t *c)
{
    if (n < 0 || j < 0 || j >= m || ld < m || S < 2 || batch_rows <= 0) return -1;
    int64_t stride = sketch_stride(n, sketch_max_rows);
    orc_entry *R = NULL;
    int64_t kR = 0;
    float *vals = (float *)malloc(sizeof(float) * (size_t)(batch_rows / stride + 2));
    if (!vals) return -1;
    for (int64_t b0 = 0; b0 < n; b0 += batch_rows) {
        int64_t b1 = b0 + batch_rows < n ? b0 + batch_rows : n, N = 0;
        for (int64_t i = (b0 + stride - 1) / stride * stride; i < b1; i += stride) {
            float x = X[i * ld + j];
            if (isnan(x)) continue;
            if (isinf(x)) {
                free(vals);
                free(R);
                return -1;
            }
            if (x == 0.0f) x = 0.0f;
            vals[N++] = x;
        }
        if (summary_add_batch(&R, &kR, vals, N, S) != ORC_OK) {
            free(vals);
            free(R);
            return -1;
        }
    }
    for (int64_t i = 0; i < kR; ++i) {
        v[i] = R[i].v;
        c[i] = R[i].c;
    }
    free(vals);
    free(R);
    return kR;
}

/* CSR input in batches of batch_rows rows: as orc_sketch_cuts_merge_dense,
 * absent entries and NaN values missing. */
int orc_sketch_cuts_merge_csr(const int64_t *indptr, const int32_t *indices, const float *values, int64_t n,
                              int32_t m, int32_t max_bin, int64_t sketch_max_rows, int32_t S, int64_t batch_rows,
                              int32_t *cut_ptr, float *cut_values, int64_t *entries_out)
{
    if (n < 0 || m <= 0 || max_bin < 2 || S < 2 || batch_rows <= 0) return ORC_EINVAL;
    int64_t stride = sketch_stride(n, sketch_max_rows);
    for (int64_t i = 0; i < n; ++i)
        for (int64_t e = indptr[i]; e < indptr[i + 1]; ++e)
            if (indices[e] < 0 || indices[e] >= m || isinf(values[e])) return ORC_EINVAL;
    orc_entry **R = (orc_entry **)calloc((size_t)m, sizeof(orc_entry *));
    int64_t *kR = (int64_t *)calloc((size_t)m, sizeof(int64_t));
    int64_t *cnt = (int64_t *)malloc(sizeof(int64_t) * (size_t)(m + 1));
    int64_t *fill = (int64_t *)malloc(sizeof(int64_t) * (size_t)m);
    float *vals = NULL;
    int rc = (R && kR && cnt && fill) ? ORC_OK : ORC_ENOMEM;
    for (int64_t b0 = 0; b0 < n && rc == ORC_OK; b0 += batch_rows) {
        int64_t b1 = b0 + batch_rows < n ? b0 + batch_rows : n;
        /* the batch's sample values, grouped by feature */
        memset(cnt, 0, sizeof(int64_t) * (size_t)(m + 1));
        for (int64_t i = (b0 + stride - 1) / stride * stride; i < b1; i += stride)
            for (int64_t e = indptr[i]; e < indptr[i + 1]; ++e)
                if (!isnan(values[e])) cnt[indices[e] + 1]++;
        for (int32_t j = 0; j < m; ++j) cnt[j + 1] += cnt[j];
        free(vals);
        vals = (float *)malloc(sizeof(float) * (size_t)(cnt[m] + 1));
        if (!vals) {
            rc = ORC_ENOMEM;
            break;
        }
        for (int32_t j = 0; j < m; ++j) fill[j] = cnt[j];
        for (int64_t i = (b0 + stride - 1) / stride * stride; i < b1; i += stride)
            for (int64_t e = indptr[i]; e < indptr[i + 1]; ++e) {
                float x = values[e];
                if (isnan(x)) continue;
                if (x == 0.0f) x = 0.0f;
                vals[fill[indices[e]]++] = x;
            }
        int oom = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : oom)
        for (int32_t j = 0; j < m; ++j)
            if (summary_add_batch(&R[j], &kR[j], vals + cnt[j], cnt[j + 1] - cnt[j], S) != ORC_OK) oom = 1;
        if (oom) rc = ORC_ENOMEM;
    }
    if (rc == ORC_OK) {
        cut_ptr[0] = 0;
        for (int32_t j = 0; j < m; ++j) {
            int32_t c = cuts_from_summary(R[j], kR[j], max_bin, cut_values + cut_ptr[j]);
            cut_ptr[j + 1] = cut_ptr[j] + c;
            if (entries_out) entries_out[j] = kR[j];
        }
    }
    if (R)
        for (int32_t j = 0; j < m; ++j) free(R[j]);
    free(R);
    free(kR);
    free(cnt);
    free(fill);
    free(vals);
    return rc;
}

/* bin(x) = #{cuts < x}: the cuts ascend, so this is the first index whose
 * cut is not below x (bisection). */
static int32_t lookup_bin(const float *cuts, int32_t nc, float x)
{
    int32_t lo = 0, hi = nc;
    while (lo < hi) {
        int32_t mid = lo + (hi - lo) / 2;
        if (cuts[mid] < x)
            lo = mid + 1;
        else
            hi = mid;
    }
    return lo;
}

/* Dense raw -> dense bins (ORC_MISSING for NaN). */
int orc_bin_dense(const float *X, int64_t n, int32_t m, int64_t ld, const int32_t *cut_ptr,
                  const float *cut_values, uint16_t *bins)
{
    int bad = 0;
#pragma omp parallel for schedule(static) reduction(| : bad)
    for (int64_t i = 0; i < n; ++i)
        for (int32_t j = 0; j < m; ++j) {
            float x = X[i * ld + j];
            if (isinf(x)) bad = 1;
            bins[i * m + j] = isnan(x) || isinf(x) ? (uint16_t)ORC_MISSING
                                                   : (uint16_t)lookup_bin(cut_values + cut_ptr[j],
                                                                          cut_ptr[j + 1] - cut_ptr[j], x);
        }
    return bad ? ORC_EINVAL : ORC_OK;
}

/* CSR raw -> CSR bins.  NaN entries are dropped (they are missing), so the
 * output row pointer can differ from the input one.  Features must be
 * strictly ascending within a row. */
int orc_bin_csr(const int64_t *indptr, const int32_t *indices, const float *values, int64_t n,
                int32_t m, const int32_t *cut_ptr, const float *cut_values, int64_t *out_indptr,
                int32_t *out_feat, uint16_t *out_bin)
{
    int64_t o = 0;
    out_indptr[0] = 0;
    for (int64_t i = 0; i < n; ++i) {
        int32_t prev = -1;
        for (int64_t e = indptr[i]; e < indptr[i + 1]; ++e) {
            int32_t j = indices[e];
            float x = values[e];
            if (j <= prev || j >= m || isinf(x)) return ORC_EINVAL;
            prev = j;
            if (isnan(x)) continue;
            out_feat[o] = j;
            out_bin[o] = (uint16_t)lookup_bin(cut_values + cut_ptr[j], cut_ptr[j + 1] - cut_ptr[j], x);
            ++o;
        }
        out_indptr[i + 1] = o;
    }
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Sec. 2.2 / Sec. 3.2: ELLPACK rows.  Reading of the layout:                */
/*  - dense: slot j holds feature j's local bin, or the null symbol          */
/*    2^w-1 when missing; w = ceil(log2(max_j B_j + has_missing)), w >= 1    */
/*  - sparse: the row's present features in ascending order, each as the     */
/*    global bin off_j + bin (off = prefix sum of B_j); padding slots hold    */
/*    the null symbol sum_j B_j; w = ceil(log2(sum_j B_j + 1))               */
/*  - a row is an LSB-first bit stream of stride*w bits in 32-bit words,      */
/*    padded with zero words to a multiple of 4 words; rows are stored one    */
/*    after another.                                                          */
/* ------------------------------------------------------------------------ */
static int32_t ceil_log2_u64(uint64_t v)
{
    int32_t b = 0;
    while (b < 64 && ((uint64_t)1 << b) < v) ++b;
    return b;
}

static int32_t ceil_log2_i64(int64_t v)
{
    return v <= 1 ? 0 : ceil_log2_u64((uint64_t)v);
}

static void put_bits(uint32_t *row, int64_t bitpos, uint32_t sym, int32_t w)
{
    for (int32_t b = 0; b < w; ++b) {
        if ((sym >> b) & 1u) {
            int64_t p = bitpos + b;
            row[p >> 5] |= 1u << (p & 31);
        }
    }
}

/* Layout parameters, in the order: w, stride, row_words, null_symbol. */
void orc_ellpack_geometry(int32_t sparse, int32_t m, const int32_t *nbins, int32_t has_missing,
                          int32_t max_row_nnz, int32_t *out4)
{
    int64_t total = 0;
    int32_t maxb = 1;
    for (int32_t j = 0; j < m; ++j) {
        total += nbins[j];
        if (nbins[j] > maxb) maxb = nbins[j];
    }
    int32_t w, stride, nullsym;
    if (sparse) {
        w = ceil_log2_u64((uint64_t)total + 1);
        stride = max_row_nnz;
        nullsym = (int32_t)total;
    } else {
        w = ceil_log2_u64((uint64_t)maxb + (has_missing ? 1 : 0));
        stride = m;
        nullsym = (int32_t)((1u << w) - 1u);
    }
    if (w < 1) w = 1;
    if (!sparse) nullsym = (int32_t)((1u << w) - 1u);
    int64_t words = ((int64_t)stride * w + 31) / 32;
    int64_t row_words = (words + 3) / 4 * 4;
    if (row_words == 0) row_words = 4;
    out4[0] = w;
    out4[1] = stride;
    out4[2] = (int32_t)row_words;
    out4[3] = nullsym;
}

/* Encode dense bins into ELLPACK rows; out has n*row_words words. */
void orc_ellpack_dense(const uint16_t *bins, int64_t n, int32_t m, int32_t w, int32_t row_words,
                       uint32_t nullsym, uint32_t *out)
{
    memset(out, 0, sizeof(uint32_t) * (size_t)(n * row_words));
    for (int64_t i = 0; i < n; ++i) {
        uint32_t *row = out + i * row_words;
        for (int32_t j = 0; j < m; ++j) {
            uint16_t b = bins[i * m + j];
            uint32_t sym = (b == ORC_MISSING) ? nullsym : (uint32_t)b;
            put_bits(row, (int64_t)j * w, sym, w);
        }
    }
}

/* Encode CSR bins into sparse ELLPACK rows. */
void orc_ellpack_csr(const int64_t *indptr, const int32_t *feat, const uint16_t *bin, int64_t n,
                     int32_t m, const int32_t *nbins, int32_t w, int32_t stride, int32_t row_words,
                     uint32_t nullsym, uint32_t *out)
{
    int64_t *off = (int64_t *)malloc(sizeof(int64_t) * (size_t)(m + 1));
    off[0] = 0;
    for (int32_t j = 0; j < m; ++j) off[j + 1] = off[j] + nbins[j];
    memset(out, 0, sizeof(uint32_t) * (size_t)(n * row_words));
    for (int64_t i = 0; i < n; ++i) {
        uint32_t *row = out + i * row_words;
        int32_t s = 0;
        for (int64_t e = indptr[i]; e < indptr[i + 1]; ++e, ++s)
            put_bits(row, (int64_t)s * w, (uint32_t)(off[feat[e]] + bin[e]), w);
        for (; s < stride; ++s) put_bits(row, (int64_t)s * w, nullsym, w);
    }
    free(off);
}

/* ------------------------------------------------------------------------ */
/* Sec. 2.1, Eq. 4-5: first and second derivatives of the loss at the       */
/* current prediction, in double precision, stored as float pairs (g, h).   */
/*   logistic: s = 1/(1+exp(-z)); g = s - y; h = max(s*(1-s), 1e-16)        */
/*   squared : g = z - y; h = 1                                             */
/* An optional per-row weight multiplies both (in double).                  */
/* ------------------------------------------------------------------------ */
int orc_gradients(int32_t loss, const float *margin, const float *label, const float *weight,
                  int64_t n, float *gpair)
{
    if (loss != ORC_LOSS_LOGISTIC && loss != ORC_LOSS_SQUARED) return ORC_EINVAL;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        double z = (double)margin[i];
        double y = (double)label[i];
        double g, h;
        if (loss == ORC_LOSS_LOGISTIC) {
            double t = orc_exp(-z);
            double s = 1.0 / (1.0 + t);
            g = s - y;
            h = s * (1.0 - s);
            if (h < 1e-16) h = 1e-16;
        } else {
            g = z - y;
            h = 1.0;
        }
        if (weight) {
            double wt = (double)weight[i];
            g = g * wt;
            h = h * wt;
        }
        gpair[2 * i] = (float)g;
        gpair[2 * i + 1] = (float)h;
    }
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Sec. 2.4, Eq. 9 and Sec. 3.4, Alg. 7: minimal variance sampling.          */
/* Rows are kept with probability proportional to the regularized gradient  */
/* magnitude r = sqrt(g^2 + lambda*h^2).  Exact integer reading:              */
/*   a_i = rint(r_i * 2^e) as int64, e = 62 - E - L, M = max r < 2^E,         */
/*         L = ceil(log2 n)                                                   */
/*   K   = max(1, rint(f*n))                                                  */
/*   T*  = least integer T >= 1 with sum_i min(1, a_i/T) <= K, i.e.           */
/*         F(T) <= (K - C(T)) * T, C(T) = #{a_i >= T}, F(T) = sum_{a_i<T} a_i  */
/*   keep i iff a_i >= T* or U_i * T* < a_i * 2^64, U_i = word (row mod 4) of */
/*         Philox4x64-10(counter = (row div 4, iteration, 0, 0),             */
/*         key = (seed, 0)): one block gives the words of four rows          */
/*   weight w_i = 1 if a_i >= T*, else T* / a_i (the inverse of the        */
/*         inclusion probability)                                            */
/* Rows with a_i = 0 are never kept (only rows with non-zero gradients stay). */
/* ------------------------------------------------------------------------ */
int orc_mvs_keys(const float *gpair, int64_t n, double mvs_lambda, int64_t *keys, int32_t *e_out)
{
    double M = 0.0;
    int bad = 0;
#pragma omp parallel for schedule(static) reduction(max : M) reduction(| : bad)
    for (int64_t i = 0; i < n; ++i) {
        double g = (double)gpair[2 * i], h = (double)gpair[2 * i + 1];
        double r = sqrt(g * g + mvs_lambda * (h * h));
        if (isnan(r) || isinf(r)) bad = 1;
        else if (r > M) M = r;
    }
    if (bad) return ORC_EINVAL;
    int E;
    frexp(M, &E); /* M < 2^E (E = 0 when M = 0) */
    int32_t e = 62 - E - ceil_log2_i64(n);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        double g = (double)gpair[2 * i], h = (double)gpair[2 * i + 1];
        double r = sqrt(g * g + mvs_lambda * (h * h));
        keys[i] = (int64_t)rint(ldexp(r, e));
    }
    *e_out = e;
    return ORC_OK;
}

int64_t orc_mvs_target(double f, int64_t n)
{
    int64_t K = (int64_t)rint(f * (double)n);
    return K < 1 ? 1 : K;
}

/* phi(T) <= K  <=>  F(T) <= (K - C(T)) * T, evaluated exactly in 128 bits */
static int threshold_ok(const int64_t *keys, int64_t n, int64_t K, int64_t T)
{
    int64_t C = 0;
    __int128 F = 0;
#pragma omp parallel
    {
        int64_t c = 0;
        __int128 f = 0;
#pragma omp for schedule(static) nowait
        for (int64_t i = 0; i < n; ++i) {
            if (keys[i] >= T)
                ++c;
            else
                f += keys[i];
        }
#pragma omp critical
        {
            C += c;
            F += f;
        }
    }
    return F <= (__int128)(K - C) * (__int128)T;
}

/* Least T >= 1 with phi(T) <= K, by bisection (phi is non-increasing). */
int64_t orc_mvs_threshold(const int64_t *keys, int64_t n, int64_t K)
{
    __int128 sum = 0;
    int64_t mx = 0;
#pragma omp parallel
    {
        __int128 s = 0;
        int64_t x = 0;
#pragma omp for schedule(static) nowait
        for (int64_t i = 0; i < n; ++i) {
            s += keys[i];
            if (keys[i] > x) x = keys[i];
        }
#pragma omp critical
        {
            sum += s;
            if (x > mx) mx = x;
        }
    }
    /* at T = hi every key is below T and sum/T <= K, so hi satisfies it */
    __int128 hi = (__int128)mx + 1;
    __int128 q = (sum + K - 1) / K;
    if (q > hi) hi = q;
    int64_t lo = 1, h = (int64_t)hi;
    while (lo < h) {
        int64_t mid = lo + (h - lo) / 2;
        if (threshold_ok(keys, n, K, mid))
            h = mid;
        else
            lo = mid + 1;
    }
    return lo;
}

uint64_t orc_mvs_uniform(uint64_t seed, uint64_t iteration, uint64_t row)
{
    uint64_t ctr[4] = {row >> 2, iteration, 0, 0}, key[2] = {seed, 0}, out[4];
    orc_philox4x64_10(ctr, key, out);
    return out[row & 3];
}

/* keep[i] = 1 when row (row_offset + i) is sampled. */
void orc_mvs_select(const int64_t *keys, int64_t n, int64_t T, uint64_t seed, uint64_t iteration,
                    int64_t row_offset, uint8_t *keep)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        int64_t a = keys[i];
        if (a >= T) {
            keep[i] = 1;
            continue;
        }
        uint64_t U = orc_mvs_uniform(seed, iteration, (uint64_t)(row_offset + i));
        keep[i] = ((unsigned __int128)U * (unsigned __int128)(uint64_t)T) <
                  ((unsigned __int128)(uint64_t)a << 64);
    }
}

double orc_mvs_weight(int64_t a, int64_t T)
{
    return a >= T ? 1.0 : (double)T / (double)a;
}

/* ------------------------------------------------------------------------ */
/* Sec. 2.3, the other two samplers (a reading: each random draw is the     */
/* row's Philox word U_i of the MVS stream, compared with a probability     */
/* scaled to 2^64; p < 1 gives the integer floor(p 2^64), p = 1 keeps all).  */
/* SGB (Friedman): each row is kept with probability f, weight 1.            */
/* GOSS (Ke et al.): the top a*100% rows by |g| -- keys k_i = rint(|g_i| 2^e) */
/* as in orc_mvs_keys with lambda = 0, A = rint(a n), every row whose key is */
/* at least the A-th largest key (ties included; none when A = 0) -- plus   */
/* each other row with probability p = b / (1 - a), b = f - a, weighted by   */
/* (1 - a) / b = 1/p.                                                        */
/* ------------------------------------------------------------------------ */
static int bernoulli(uint64_t U, double p)
{
    if (p >= 1.0) return 1;
    return U < (uint64_t)ldexp(p, 64);
}

void orc_sgb_select(int64_t n, double f, uint64_t seed, uint64_t iteration, int64_t row_offset, uint8_t *keep)
{
    for (int64_t i = 0; i < n; ++i)
        keep[i] = (uint8_t)bernoulli(orc_mvs_uniform(seed, iteration, (uint64_t)(row_offset + i)), f);
}

static int cmp_i64_desc(const void *a, const void *b)
{
    int64_t x = *(const int64_t *)a, y = *(const int64_t *)b;
    return x < y ? 1 : (x > y ? -1 : 0);
}

/* The top threshold: the A-th largest key, or INT64_MAX when A = 0. */
int64_t orc_goss_top_threshold(const int64_t *keys, int64_t n, int64_t A)
{
    if (A <= 0 || n <= 0) return INT64_MAX;
    if (A > n) A = n;
    int64_t *s = (int64_t *)malloc(sizeof(int64_t) * (size_t)n);
    memcpy(s, keys, sizeof(int64_t) * (size_t)n);
    qsort(s, (size_t)n, sizeof(int64_t), cmp_i64_desc);
    int64_t t = s[A - 1];
    free(s);
    return t;
}

int64_t orc_goss_top_count(double a, int64_t n)
{
    int64_t A = (int64_t)rint(a * (double)n);
    return A < 0 ? 0 : (A > n ? n : A);
}

void orc_goss_select(const int64_t *keys, int64_t n, int64_t T_top, double a, double b, uint64_t seed,
                     uint64_t iteration, int64_t row_offset, uint8_t *keep)
{
    const double p = b / (1.0 - a);
    for (int64_t i = 0; i < n; ++i)
        keep[i] = (uint8_t)(keys[i] >= T_top ||
                            bernoulli(orc_mvs_uniform(seed, iteration, (uint64_t)(row_offset + i)), p));
}

double orc_goss_weight(int64_t key, int64_t T_top, double a, double b)
{
    return key >= T_top ? 1.0 : (1.0 - a) / b;
}

/* ------------------------------------------------------------------------ */
/* Exact integer gradient sums.  Over the R training rows:                   */
/*   M = max |x| < 2^E, e = 62 - E - ceil(log2 R), q = rint(x * 2^e) (int64)  */
/* so any sum of R values stays below 2^62 in magnitude.  Sums go back to    */
/* double as ldexp((double)Q, -e).                                           */
/* ------------------------------------------------------------------------ */
static int32_t fx_exponent(const double *x, int64_t R, int64_t stride)
{
    double M = 0.0;
#pragma omp parallel for schedule(static) reduction(max : M)
    for (int64_t i = 0; i < R; ++i) {
        double a = fabs(x[i * stride]);
        if (a > M) M = a;
    }
    int E;
    frexp(M, &E);
    return 62 - E - ceil_log2_i64(R);
}

void orc_fixed_point(const double *gw, int64_t R, int64_t *q, int32_t *e_g, int32_t *e_h)
{
    int32_t eg = fx_exponent(gw, R, 2), eh = fx_exponent(gw + 1, R, 2);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < R; ++i) {
        q[2 * i] = (int64_t)rint(ldexp(gw[2 * i], eg));
        q[2 * i + 1] = (int64_t)rint(ldexp(gw[2 * i + 1], eh));
    }
    *e_g = eg;
    *e_h = eh;
}

/* ------------------------------------------------------------------------ */
/* Alg. 1 BuildHistograms: for one node, sum (q_g, q_h) of its rows into    */
/* hist[off_j + bin][2] for every present (feature, bin).  Missing values    */
/* contribute nothing.  hist must hold (sum_j B_j)*2 int64 and is zeroed.   */
/* rows[] are row ids of d; q is indexed by the same ids.                     */
/* ------------------------------------------------------------------------ */
static int64_t total_bins(const orc_data *d, int64_t *off)
{
    int64_t t = 0;
    for (int32_t j = 0; j < d->m; ++j) {
        if (off) off[j] = t;
        t += d->nbins[j];
    }
    if (off) off[d->m] = t;
    return t;
}

void orc_build_hist(const orc_data *d, const int64_t *rows, int64_t n_rows, const int64_t *q,
                    int64_t *hist)
{
    int64_t *off = (int64_t *)malloc(sizeof(int64_t) * (size_t)(d->m + 1));
    int64_t tb = total_bins(d, off);
    memset(hist, 0, sizeof(int64_t) * (size_t)(2 * tb));
    /* omp: each thread sums its rows into a histogram of its own, then the
     * integer histograms are added (exact, so the order does not matter) */
#pragma omp parallel if (n_rows >= 4096)
    {
        int64_t *h = hist;
#ifdef _OPENMP
        h = (int64_t *)calloc((size_t)(2 * tb + 2), sizeof(int64_t));
#endif
#pragma omp for schedule(static) nowait
        for (int64_t k = 0; k < n_rows; ++k) {
            int64_t r = rows[k];
            int64_t qg = q[2 * r], qh = q[2 * r + 1];
            if (d->dense) {
                for (int32_t j = 0; j < d->m; ++j) {
                    uint16_t b = d->dense[r * d->m + j];
                    if (b == ORC_MISSING) continue;
                    h[2 * (off[j] + b)] += qg;
                    h[2 * (off[j] + b) + 1] += qh;
                }
            } else {
                for (int64_t e = d->indptr[r]; e < d->indptr[r + 1]; ++e) {
                    int64_t gb = off[d->feat[e]] + d->bin[e];
                    h[2 * gb] += qg;
                    h[2 * gb + 1] += qh;
                }
            }
        }
#ifdef _OPENMP
#pragma omp critical
        for (int64_t t = 0; t < 2 * tb; ++t) hist[t] += h[t];
        free(h);
#endif
    }
    free(off);
}

/* ------------------------------------------------------------------------ */
/* Alg. 1 EvaluateSplit with the loss reduction of Eq. 8:                    */
/*   gain = 1/2 [G_L^2/(H_L+lambda) + G_R^2/(H_R+lambda) - G^2/(H+lambda)]   */
/*          - gamma                                                          */
/* For every feature j with B_j >= 2, every s in 1..B_j-1 and both           */
/* directions for missing values (right first, then left):                   */
/*   Q_L = sum_{b<s} H_j[b] (+ missing sums if missing goes left)            */
/*   Q_R = node sum - Q_L                                                    */
/* A candidate is valid when H_L >= mcw and H_R >= mcw and its gain is not   */
/* NaN.  The best is the highest gain; ties keep the earliest candidate in   */
/* (feature, s, direction) order.                                            */
/* ------------------------------------------------------------------------ */
static double to_double(int64_t Q, int32_t e)
{
    return ldexp((double)Q, -e);
}

static double split_gain(double GL, double HL, double GR, double HR, double G, double H,
                         double lambda, double gamma)
{
    double a = (GL * GL) / (HL + lambda);
    double b = (GR * GR) / (HR + lambda);
    double c = (G * G) / (H + lambda);
    return 0.5 * ((a + b) - c) - gamma;
}

/* The best candidate of one feature (the first of the highest gain in
 * (s, direction) order); valid = 0 when it has none. */
static orc_split eval_feature(const int64_t *hj, int32_t j, int32_t B, const int64_t node_sum[2], double G,
                              double H, const orc_params *p, int32_t e_g, int32_t e_h)
{
    orc_split best;
    memset(&best, 0, sizeof(best));
    best.feature = -1;
    best.split_bin = -1;
    if (B < 2) return best;
    int64_t tg = 0, th = 0;
    for (int32_t b = 0; b < B; ++b) {
        tg += hj[2 * b];
        th += hj[2 * b + 1];
    }
    int64_t miss_g = node_sum[0] - tg, miss_h = node_sum[1] - th;
    int64_t lg = 0, lh = 0;
    for (int32_t s = 1; s < B; ++s) {
        lg += hj[2 * (s - 1)];
        lh += hj[2 * (s - 1) + 1];
        for (int32_t dir = 0; dir < 2; ++dir) {
            int64_t QLg = lg + (dir ? miss_g : 0), QLh = lh + (dir ? miss_h : 0);
            int64_t QRg = node_sum[0] - QLg, QRh = node_sum[1] - QLh;
            double GL = to_double(QLg, e_g), HL = to_double(QLh, e_h);
            double GR = to_double(QRg, e_g), HR = to_double(QRh, e_h);
            if (!(HL >= p->min_child_weight && HR >= p->min_child_weight)) continue;
            double gain = split_gain(GL, HL, GR, HR, G, H, p->lambda, p->gamma);
            if (isnan(gain)) continue;
            if (!best.valid || gain > best.gain) {
                best.valid = 1;
                best.gain = gain;
                best.feature = j;
                best.split_bin = s;
                best.default_left = dir;
                best.left_g = QLg;
                best.left_h = QLh;
                best.right_g = QRg;
                best.right_h = QRh;
            }
        }
    }
    return best;
}

void orc_eval_node(const int64_t *hist, const int64_t node_sum[2], const int32_t *nbins, int32_t m,
                   const orc_params *p, int32_t e_g, int32_t e_h, orc_split *out)
{
    double G = to_double(node_sum[0], e_g), H = to_double(node_sum[1], e_h);
    int64_t *off = (int64_t *)malloc(sizeof(int64_t) * (size_t)(m + 1));
    orc_split *per = (orc_split *)malloc(sizeof(orc_split) * (size_t)(m + 1));
    off[0] = 0;
    for (int32_t j = 0; j < m; ++j) off[j + 1] = off[j] + nbins[j];
    /* omp: features are independent */
#pragma omp parallel for schedule(dynamic, 4) if (off[m] >= 4096)
    for (int32_t j = 0; j < m; ++j)
        per[j] = eval_feature(hist + 2 * off[j], j, nbins[j], node_sum, G, H, p, e_g, e_h);
    /* the first candidate of the highest gain in (feature, s, direction)
     * order: features in order, strictly higher gains only */
    orc_split best;
    memset(&best, 0, sizeof(best));
    best.feature = -1;
    best.split_bin = -1;
    for (int32_t j = 0; j < m; ++j)
        if (per[j].valid && (!best.valid || per[j].gain > best.gain)) best = per[j];
    free(off);
    free(per);
    *out = best;
}

/* Bin of (row, feature) in d, or -1 when missing. */
static int32_t row_bin(const orc_data *d, int64_t r, int32_t j)
{
    if (d->dense) {
        uint16_t b = d->dense[r * d->m + j];
        return b == ORC_MISSING ? -1 : (int32_t)b;
    }
    for (int64_t e = d->indptr[r]; e < d->indptr[r + 1]; ++e)
        if (d->feat[e] == j) return d->bin[e];
    return -1;
}

/* Alg. 1 RepartitionInstances: a row goes left iff its bin for the split
 * feature is below split_bin, or it is missing and default_left is set.
 * Stable: both sides keep the input order.  Returns the left count. */
int64_t orc_partition(const orc_data *d, const int64_t *rows, int64_t n_rows, int32_t feature,
                      int32_t split_bin, int32_t default_left, int64_t *out)
{
    int64_t nl = 0;
    for (int64_t k = 0; k < n_rows; ++k) {
        int32_t b = row_bin(d, rows[k], feature);
        int left = (b < 0) ? default_left : (b < split_bin);
        if (left) out[nl++] = rows[k];
    }
    int64_t nr = nl;
    for (int64_t k = 0; k < n_rows; ++k) {
        int32_t b = row_bin(d, rows[k], feature);
        int left = (b < 0) ? default_left : (b < split_bin);
        if (!left) out[nr++] = rows[k];
    }
    return nl;
}

/* Sec. 2.4 (MVS): lambda estimated from the data as the square of the      */
/* initial leaf value, read as the unregularized Newton step of all n rows  */
/* at the given margins: gradients (Eq. 4-5), their fixed point over the n  */
/* rows, G and H the exact integer sums, w0 = -G/H, lambda = w0^2 (0 when H */
/* is 0).                                                                    */
double orc_mvs_lambda_estimate(int32_t loss, const float *margin, const float *label, int64_t n)
{
    if (n <= 0) return 0.0;
    float *gp = (float *)malloc((size_t)n * 2 * sizeof(float));
    double *gw = (double *)malloc((size_t)n * 2 * sizeof(double));
    int64_t *q = (int64_t *)malloc((size_t)n * 2 * sizeof(int64_t));
    double lam = 0.0;
    if (gp && gw && q && orc_gradients(loss, margin, label, NULL, n, gp) == 0) {
        for (int64_t i = 0; i < 2 * n; ++i) gw[i] = (double)gp[i];
        int32_t eg, eh;
        orc_fixed_point(gw, n, q, &eg, &eh);
        int64_t G = 0, H = 0;
        for (int64_t i = 0; i < n; ++i) {
            G += q[2 * i];
            H += q[2 * i + 1];
        }
        if (H != 0) {
            double w0 = -to_double(G, eg) / to_double(H, eh);
            lam = w0 * w0;
        }
    } else {
        lam = -1.0;
    }
    free(gp);
    free(gw);
    free(q);
    return lam;
}

/* Eq. 6, scaled by the learning rate: leaf = (float)((-G/(H+lambda)) * eta) */
float orc_leaf_value(int64_t Qg, int64_t Qh, int32_t e_g, int32_t e_h, double lambda, double eta)
{
    double G = to_double(Qg, e_g), H = to_double(Qh, e_h);
    double w = -G / (H + lambda);
    return (float)(w * eta);
}

/* Leaf reached by row r of d in a heap-ordered tree. */
static int64_t leaf_of_binned(const orc_data *d, int64_t r, const orc_node *tree)
{
    int64_t id = 0;
    while (!(tree[id].flags & ORC_NODE_LEAF)) {
        int32_t b = row_bin(d, r, tree[id].feature);
        int left = (b < 0) ? ((tree[id].flags & ORC_NODE_DEFAULT_LEFT) != 0) : (b < tree[id].split_bin);
        id = left ? 2 * id + 1 : 2 * id + 2;
    }
    return id;
}

/* ------------------------------------------------------------------------ */
/* One boosting iteration: Alg. 7 (sample, compact) then Alg. 1 (in-core    */
/* tree construction) grown level by level, then the margin update of      */
/* Eq. 1 for all n rows.  The tree is heap ordered: the children of node i  */
/* are 2i+1 and 2i+2, and tree[] has 2^(max_depth+1)-1 entries.             */
/* Optional outputs: sel (the R sampled rows, ascending), q (their 2R        */
/* fixed-point gradients), gpair_out (the n float gradient pairs).           */
/* ------------------------------------------------------------------------ */
int orc_train_tree(const orc_data *d, const float *label, float *margin, const orc_params *p,
                   orc_node *tree, orc_info *info, int64_t *sel, int64_t *q_out, float *gpair_out)
{
    int64_t n = d->n;
    int32_t D = p->max_depth;
    if (D < 0 || D > 20 || !(p->f > 0.0 && p->f <= 1.0)) return ORC_EINVAL;
    int64_t n_nodes = ((int64_t)1 << (D + 1)) - 1;
    memset(tree, 0, sizeof(orc_node) * (size_t)n_nodes);
    memset(info, 0, sizeof(*info));
    info->n_nodes = (int32_t)n_nodes;

    float *gpair = (float *)malloc(sizeof(float) * (size_t)(2 * n + 2));
    int64_t *grow = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n + 1)); /* training row -> d row */
    double *gw = (double *)malloc(sizeof(double) * (size_t)(2 * n + 2));
    if (!gpair || !grow || !gw) return ORC_ENOMEM;
    int rc = orc_gradients(p->loss, margin, label, NULL, n, gpair);
    if (rc) return rc;
    if (gpair_out) memcpy(gpair_out, gpair, sizeof(float) * (size_t)(2 * n));

    /* Alg. 7: g' <- Sample(g); compact the kept rows in ascending order */
    int64_t R = 0;
    if (p->f < 1.0) {
        int64_t *keys = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n + 1));
        uint8_t *keep = (uint8_t *)malloc((size_t)n + 1);
        if (!keys || !keep) return ORC_ENOMEM;
        const double ga = p->goss_a, gb = p->f - p->goss_a;
        if (p->sampler == ORC_SAMPLE_SGB) {
            orc_sgb_select(n, p->f, p->seed, p->iteration, 0, keep);
        } else if (p->sampler == ORC_SAMPLE_GOSS) {
            if (!(ga >= 0.0 && ga < 1.0 && gb > 0.0)) return ORC_EINVAL;
            rc = orc_mvs_keys(gpair, n, 0.0, keys, &info->e_key);
            if (rc) return rc;
            info->K = orc_goss_top_count(ga, n);
            info->T = orc_goss_top_threshold(keys, n, info->K);
            orc_goss_select(keys, n, info->T, ga, gb, p->seed, p->iteration, 0, keep);
        } else {
            rc = orc_mvs_keys(gpair, n, p->mvs_lambda, keys, &info->e_key);
            if (rc) return rc;
            info->K = orc_mvs_target(p->f, n);
            info->T = orc_mvs_threshold(keys, n, info->K);
            orc_mvs_select(keys, n, info->T, p->seed, p->iteration, 0, keep);
        }
        for (int64_t i = 0; i < n; ++i) {
            if (!keep[i]) continue;
            double w = p->sampler == ORC_SAMPLE_SGB    ? 1.0
                       : p->sampler == ORC_SAMPLE_GOSS ? orc_goss_weight(keys[i], info->T, ga, gb)
                                                       : orc_mvs_weight(keys[i], info->T);
            grow[R] = i;
            gw[2 * R] = (double)gpair[2 * i] * w;
            gw[2 * R + 1] = (double)gpair[2 * i + 1] * w;
            ++R;
        }
        free(keys);
        free(keep);
    } else {
        for (int64_t i = 0; i < n; ++i) {
            grow[i] = i;
            gw[2 * i] = (double)gpair[2 * i];
            gw[2 * i + 1] = (double)gpair[2 * i + 1];
        }
        R = n;
    }
    info->n_sampled = R;
    if (sel) memcpy(sel, grow, sizeof(int64_t) * (size_t)R);

    /* exact integer gradients of the training rows, indexed by d row id */
    int64_t *qt = (int64_t *)malloc(sizeof(int64_t) * (size_t)(2 * R + 2));
    int64_t *q = (int64_t *)calloc((size_t)(2 * n + 2), sizeof(int64_t));
    if (!qt || !q) return ORC_ENOMEM;
    orc_fixed_point(gw, R, qt, &info->e_g, &info->e_h);
    for (int64_t k = 0; k < R; ++k) {
        q[2 * grow[k]] = qt[2 * k];
        q[2 * grow[k] + 1] = qt[2 * k + 1];
    }
    if (q_out) memcpy(q_out, qt, sizeof(int64_t) * (size_t)(2 * R));

    /* Alg. 1, level by level.  The node rows are segments of one list of d
     * row ids; a split rewrites its segment as [left | right]. */
    int64_t tb = total_bins(d, NULL);
    int64_t *hist = (int64_t *)malloc(sizeof(int64_t) * (size_t)(2 * tb + 2));
    int64_t *rows = (int64_t *)malloc(sizeof(int64_t) * (size_t)(R + 1));
    int64_t *tmp = (int64_t *)malloc(sizeof(int64_t) * (size_t)(R + 1));
    int64_t *seg_b = (int64_t *)calloc((size_t)n_nodes, sizeof(int64_t));
    int64_t *seg_e = (int64_t *)calloc((size_t)n_nodes, sizeof(int64_t));
    if (!hist || !rows || !tmp || !seg_b || !seg_e) return ORC_ENOMEM;
    for (int64_t k = 0; k < R; ++k) rows[k] = grow[k];

    /* InitRoot: the root holds every training row; its sums are a direct
     * reduction */
    int64_t sg = 0, sh = 0;
#pragma omp parallel for schedule(static) reduction(+ : sg, sh)
    for (int64_t k = 0; k < R; ++k) {
        sg += qt[2 * k];
        sh += qt[2 * k + 1];
    }
    tree[0].flags = ORC_NODE_PRESENT;
    tree[0].sum_g = sg;
    tree[0].sum_h = sh;
    seg_b[0] = 0;
    seg_e[0] = R;

    for (int32_t depth = 0; depth <= D; ++depth) {
        int64_t first = ((int64_t)1 << depth) - 1, last = ((int64_t)1 << (depth + 1)) - 1;
        for (int64_t id = first; id < last; ++id) {
            orc_node *nd = &tree[id];
            if (!(nd->flags & ORC_NODE_PRESENT)) continue;
            int64_t b = seg_b[id], e = seg_e[id];
            nd->n_rows = (int32_t)(e - b);
            nd->feature = -1;
            nd->split_bin = -1;
            if (depth < D) {
                orc_build_hist(d, rows + b, e - b, q, hist);
                int64_t ns[2] = {nd->sum_g, nd->sum_h};
                orc_split s;
                orc_eval_node(hist, ns, d->nbins, d->m, p, info->e_g, info->e_h, &s);
                if (s.valid && s.gain > 0.0) {
                    int64_t nl = orc_partition(d, rows + b, e - b, s.feature, s.split_bin,
                                               s.default_left, tmp);
                    memcpy(rows + b, tmp, sizeof(int64_t) * (size_t)(e - b));
                    nd->feature = s.feature;
                    nd->split_bin = s.split_bin;
                    nd->threshold = d->cut_values[d->cut_ptr[s.feature] + s.split_bin - 1];
                    nd->gain = s.gain;
                    if (s.default_left) nd->flags |= ORC_NODE_DEFAULT_LEFT;
                    orc_node *L = &tree[2 * id + 1], *Rn = &tree[2 * id + 2];
                    L->flags = Rn->flags = ORC_NODE_PRESENT;
                    L->sum_g = s.left_g;
                    L->sum_h = s.left_h;
                    Rn->sum_g = s.right_g;
                    Rn->sum_h = s.right_h;
                    seg_b[2 * id + 1] = b;
                    seg_e[2 * id + 1] = b + nl;
                    seg_b[2 * id + 2] = b + nl;
                    seg_e[2 * id + 2] = e;
                    continue;
                }
            }
            nd->flags |= ORC_NODE_LEAF;
            nd->leaf_value =
                orc_leaf_value(nd->sum_g, nd->sum_h, info->e_g, info->e_h, p->lambda, p->eta);
        }
    }

    /* Eq. 1: every one of the n rows adds its leaf to its margin */
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        int64_t id = leaf_of_binned(d, i, tree);
        margin[i] = margin[i] + tree[id].leaf_value;
    }

    free(gpair);
    free(grow);
    free(gw);
    free(qt);
    free(q);
    free(hist);
    free(rows);
    free(tmp);
    free(seg_b);
    free(seg_e);
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Eq. 1: prediction = base + sum over trees of the reached leaf, added in   */
/* float in tree order.  Trees are concatenated heap arrays; tree t spans    */
/* nodes[offsets[t] .. offsets[t+1]).                                        */
/* ------------------------------------------------------------------------ */
void orc_predict_binned(const orc_data *d, const orc_node *nodes, const int64_t *offsets,
                        int32_t n_trees, float base, float *out)
{
    for (int64_t i = 0; i < d->n; ++i) {
        float acc = base;
        for (int32_t t = 0; t < n_trees; ++t) {
            const orc_node *tree = nodes + offsets[t];
            acc = acc + tree[leaf_of_binned(d, i, tree)].leaf_value;
        }
        out[i] = acc;
    }
}

static int64_t leaf_of_raw(const orc_node *tree, const float *x_dense, const int32_t *idx,
                           const float *val, int64_t nnz)
{
    int64_t id = 0;
    while (!(tree[id].flags & ORC_NODE_LEAF)) {
        int32_t j = tree[id].feature;
        float x = NAN;
        if (x_dense) {
            x = x_dense[j];
        } else {
            for (int64_t e = 0; e < nnz; ++e)
                if (idx[e] == j) {
                    x = val[e];
                    break;
                }
        }
        int left = isnan(x) ? ((tree[id].flags & ORC_NODE_DEFAULT_LEFT) != 0) : (x <= tree[id].threshold);
        id = left ? 2 * id + 1 : 2 * id + 2;
    }
    return id;
}

void orc_predict_raw_dense(const float *X, int64_t n, int64_t ld, const orc_node *nodes,
                           const int64_t *offsets, int32_t n_trees, float base, float *out)
{
    for (int64_t i = 0; i < n; ++i) {
        float acc = base;
        for (int32_t t = 0; t < n_trees; ++t) {
            const orc_node *tree = nodes + offsets[t];
            acc = acc + tree[leaf_of_raw(tree, X + i * ld, NULL, NULL, 0)].leaf_value;
        }
        out[i] = acc;
    }
}

void orc_predict_raw_csr(const int64_t *indptr, const int32_t *indices, const float *values,
                         int64_t n, const orc_node *nodes, const int64_t *offsets, int32_t n_trees,
                         float base, float *out)
{
    for (int64_t i = 0; i < n; ++i) {
        float acc = base;
        for (int32_t t = 0; t < n_trees; ++t) {
            const orc_node *tree = nodes + offsets[t];
            int64_t id = leaf_of_raw(tree, NULL, indices + indptr[i], values + indptr[i],
                                     indptr[i + 1] - indptr[i]);
            acc = acc + tree[id].leaf_value;
        }
        out[i] = acc;
    }
}
