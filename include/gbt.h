/*
 * gbt.h -- C-ABI of libgbt.so: the per-iteration hot path of out-of-core GPU
 * gradient boosting (Ou, "Out-of-Core GPU Gradient Boosting", KDD 2020) as
 * hand-written HIP kernels for MI355X (gfx950).
 *
 * Conventions
 *  - Every call returns gbt_status: GBT_OK (0) or a negative error.  No call
 *    aborts or throws across this boundary.  gbt_last_error() returns the
 *    message of the calling thread's last failed call.
 *  - Pointers ending in _d are device pointers on the context's device; _h
 *    are host pointers.  Arrays the caller sees are caller-allocated (for
 *    example torch tensors passed by data_ptr()); opaque objects (gbt_ctx,
 *    gbt_matrix, gbt_sampled, gbt_quantizer) are library-owned and released
 *    by their *_free / *_destroy call.
 *  - Work is enqueued on the context's stream.  Calls that return host
 *    values (counts, trees, info) synchronise that stream before returning.
 *    A context is used by one thread at a time; separate contexts are
 *    independent.
 *  - Hyperparameters are double; sizes are int64_t.
 *
 * Error codes
 *  GBT_E_INVALID      bad argument: NULL pointer, n < 0, max_bin outside
 *                     [2, 65535], f outside (0, 1], +-inf in the input,
 *                     unsorted CSR indices, an inconsistent page/matrix
 *  GBT_E_OOM          device or pinned-host allocation failed
 *  GBT_E_BUDGET       the context's device byte budget would be exceeded
 *                     (the out-of-memory limit of the paper's Table 1)
 *  GBT_E_DEVICE       a HIP runtime error (message saved)
 *  GBT_E_UNSUPPORTED  a valid request this build does not implement (for
 *                     example max_bin above the bins of one histogram group)
 *  GBT_E_IO           a page file could not be created, written or read
 */
#ifndef GBT_H
#define GBT_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t gbt_status;

#define GBT_OK 0
#define GBT_E_INVALID (-1)
#define GBT_E_OOM (-2)
#define GBT_E_BUDGET (-3)
#define GBT_E_DEVICE (-4)
#define GBT_E_UNSUPPORTED (-5)
#define GBT_E_IO (-6)

/* Samplers (Sec. 2.3 and 2.4). */
#define GBT_SAMPLE_MVS 0  /* minimal variance sampling, Eq. 9 */
#define GBT_SAMPLE_SGB 1  /* stochastic gradient boosting: uniform rows */
#define GBT_SAMPLE_GOSS 2 /* gradient-based one-side sampling */

#define GBT_ABI_VERSION 7

enum { GBT_INPUT_DENSE_F32 = 0, GBT_INPUT_CSR_F32 = 1 };
enum { GBT_LOC_HOST = 0, GBT_LOC_DEVICE = 1 };
enum { GBT_HOME_DEVICE = 0, GBT_HOME_PINNED_HOST = 1, GBT_HOME_DISK = 2 };
enum { GBT_LOSS_LOGISTIC = 0, GBT_LOSS_SQUARED = 1 };
enum { GBT_NODE_PRESENT = 1, GBT_NODE_LEAF = 2, GBT_NODE_DEFAULT_LEFT = 4 };

typedef struct gbt_ctx gbt_ctx;
typedef struct gbt_matrix gbt_matrix;
typedef struct gbt_sampled gbt_sampled;
typedef struct gbt_quantizer gbt_quantizer;

/* Raw training examples X (Sec. 2.1): dense row-major float32 with NaN for
 * a missing value, or CSR float32 whose absent entries (and NaN values) are
 * missing.  CSR column indices must be strictly ascending within a row. */
typedef struct {
    int32_t kind;          /* GBT_INPUT_DENSE_F32 | GBT_INPUT_CSR_F32 */
    int32_t location;      /* GBT_LOC_HOST | GBT_LOC_DEVICE */
    int64_t n_rows;
    int32_t n_cols;
    int32_t pad0;
    const float *values;   /* dense: n_rows*ld; CSR: nnz values */
    int64_t ld;            /* dense leading dimension (>= n_cols) */
    const int64_t *indptr; /* CSR: n_rows+1 */
    const int32_t *indices;/* CSR: nnz */
    int64_t nnz;
} gbt_input;

typedef struct {
    int32_t max_bin;          /* Sec. 2.2: bins per feature, default 256; at most 2560
                                 for dense input and 10176 for CSR input (the bins one
                                 histogram group holds), else GBT_E_UNSUPPORTED */
    int32_t page_home;        /* GBT_HOME_DEVICE | GBT_HOME_PINNED_HOST | GBT_HOME_DISK */
    int64_t sketch_max_rows;  /* 0 = 2^24: above it, every ceil(n/this)-th row is sketched */
    int64_t page_rows;        /* rows per ELLPACK page; 0 = one page */
    const char *page_dir;     /* GBT_HOME_DISK: an existing directory for the page files */
    int32_t sketch_summary;   /* 0: exact cuts of the sketch sample held whole on the device;
                                 S in [2, 2^20]: Alg. 3's merged sketch, at most S entries per
                                 feature (see gbt_quantize) */
    int32_t pad0;
} gbt_quant_params;

/* Geometry of a quantized matrix.  Symbols: dense pages hold feature j's
 * local bin in slot j (null = 2^w - 1 when any value is missing); sparse
 * pages hold the row's present features in ascending order as global bins
 * off_j + bin, padded with null = total_bins.  A row is an LSB-first bit
 * stream of stride*w bits in row_words 32-bit words (a multiple of 4). */
typedef struct {
    int64_t n_rows;
    int32_t n_cols;
    int32_t sparse;
    int32_t has_missing;
    int32_t symbol_bits;
    int32_t stride;
    int32_t row_words;
    uint32_t null_symbol;
    int32_t n_pages;
    int64_t total_bins;
    int64_t page_rows;
    int32_t page_home;
    int32_t pad0;
} gbt_matrix_info;

typedef struct {
    int32_t loss;             /* GBT_LOSS_* */
    int32_t max_depth;        /* 0..20 */
    double eta;               /* learning rate */
    double lambda;            /* L2 term of Eq. 2-3 */
    double gamma;             /* per-leaf term of Eq. 2-3 / Eq. 8 */
    double min_child_weight;  /* minimum hessian sum per child */
    double f;                 /* sampling fraction, (0, 1]; 1 = no sampling */
    double mvs_lambda;        /* lambda of Eq. 9 */
    uint64_t seed;
    uint64_t iteration;       /* tree index; keys the sampling stream */
    int32_t sampler;          /* GBT_SAMPLE_*: the sampler used when f < 1 */
    int32_t pad0;
    double goss_a;            /* GBT_SAMPLE_GOSS: the top fraction a (rest f - a) */
} gbt_train_params;

/* A node's row segment rows[begin, end) and its histogram slot. */
typedef struct {
    int32_t node_slot;
    int32_t pad0;
    int64_t begin;
    int64_t end;
} gbt_seg;

/* hist[target_slot] = parent_hist[parent_slot] - hist[built_slot] */
typedef struct {
    int32_t parent_slot;
    int32_t built_slot;
    int32_t target_slot;
    int32_t pad0;
} gbt_sub;

typedef struct {
    double gain;
    int64_t left_g, left_h, right_g, right_h; /* fixed-point sums */
    int32_t feature;
    int32_t split_bin;     /* left iff bin < split_bin */
    int32_t default_left;  /* missing values go left */
    int32_t valid;
    float threshold;       /* raw-value form: left iff x <= threshold, the cut
                              value below bin split_bin (0 when not valid) */
    int32_t pad0;
} gbt_split;

/* One node of a heap-ordered tree: the children of node i are 2i+1, 2i+2. */
typedef struct {
    int32_t feature;       /* split nodes; -1 otherwise */
    int32_t split_bin;
    float threshold;       /* raw-value form: left iff x <= threshold */
    float leaf_value;      /* leaves */
    double gain;           /* split nodes */
    int64_t sum_g, sum_h;  /* fixed-point gradient sums of the node */
    int32_t n_rows;        /* training rows in the node */
    uint8_t flags;         /* GBT_NODE_* */
    uint8_t pad[3];
} gbt_node;

/* Caller-allocated host tree of n_nodes = 2^(max_depth+1) - 1 nodes.  The
 * fixed-point exponents convert node sums back: G = sum_g * 2^-exp_g. */
typedef struct {
    int32_t max_depth;
    int32_t n_nodes;
    int32_t exp_g;
    int32_t exp_h;
    gbt_node *nodes;
} gbt_tree;

typedef struct {
    int64_t n_sampled;      /* R: rows the tree was built on */
    int64_t threshold;      /* MVS threshold T* (0 without sampling) */
    int32_t exp_key;        /* MVS key exponent */
    int32_t hist_launches;  /* histogram-building kernel launches */
    int64_t hist_rows;      /* rows streamed by the histogram kernels */
    int64_t hist_updates;   /* non-null (row, feature) updates performed */
    int64_t hist_bytes;     /* algorithmic bytes of the histogram kernels */
    /* kernel time per phase, from HIP events on the context stream (timing on) */
    double ms_hist;         /* histogram-building kernel */
    double ms_hist_aux;     /* histogram zeroing and sibling subtraction */
    double ms_sample;       /* gradients, sampling, compaction, fixed point */
    double ms_split;        /* split evaluation and partitioning */
    double ms_margin;       /* leaves and the margin update */
    double ms_total;        /* wall time of the call */
    double h2d_bytes;       /* bytes streamed from pinned-host or disk pages */
    int32_t hist_kernel;    /* GBT_HIST_PLAIN or GBT_HIST_ROTATED (dense), 0 sparse */
    int32_t hist_cols;      /* bytes per symbol (1 or 2) of the partition's column copy of
                               the training page when the root histogram pass also wrote it
                               (counted in hist_bytes); 0: a kernel of its own did or none
                               was made */
} gbt_tree_stats;

typedef struct {
    double f;
    double mvs_lambda;
    uint64_t seed;
    uint64_t iteration;
    int32_t loss;           /* used when gradients are recomputed from margins */
    int32_t sampler;        /* GBT_SAMPLE_* */
    double goss_a;          /* GBT_SAMPLE_GOSS: the top fraction a (rest f - a) */
} gbt_sample_params;

typedef struct {
    int64_t n_sampled;
    int64_t threshold;      /* MVS: T*; GOSS: the top threshold t; SGB: 0 */
    int64_t target;         /* MVS: K = max(1, rint(f*n)); GOSS: A; SGB: 0 */
    int32_t exp_key;
    int32_t exp_g;
    int32_t exp_h;
    int32_t is_alias;       /* f = 1: the page is the data's own page */
    const uint32_t *page_d; /* R rows of row_words words */
    const int32_t *rows_d;  /* R global row ids, ascending */
    const double *gpair_d;  /* R reweighted (g', h') in double */
    const int64_t *gpair_fx_d; /* R fixed-point (q_g, q_h) */
} gbt_sampled_info;

/* ---- library ----------------------------------------------------------- */
int32_t gbt_abi_version(void);
const char *gbt_last_error(void);

/* ---- context ------------------------------------------------------------
 * device: HIP device ordinal.  budget_bytes: cap on library-owned device
 * allocations (0 = unlimited).  hip_stream: the stream work is enqueued on
 * (NULL = the device's null stream).  A second stream at default priority
 * is created for host-to-device page copies. */
gbt_status gbt_ctx_create(int32_t device, uint64_t budget_bytes, void *hip_stream, gbt_ctx **out);
/* Releases the context.  Every matrix, quantizer and sampled set made on it
 * must be freed first: they hold device memory of the context and refer to
 * it. */
gbt_status gbt_ctx_destroy(gbt_ctx *ctx);
/* Bytes of device memory the context currently holds (budgeted). */
gbt_status gbt_ctx_memory(gbt_ctx *ctx, uint64_t *used_bytes, uint64_t *peak_bytes);
/* HIP events on the context stream (gbt_tree_stats.ms_*): 0 off, 1 around
 * the histogram-building kernel only, 2 around every phase. */
gbt_status gbt_ctx_set_timing(gbt_ctx *ctx, int32_t level);
/* Which dense histogram kernel the context uses (results are identical):
 * GBT_HIST_AUTO chooses by pass size, GBT_HIST_PLAIN forces one lane per row
 * over a feature's contiguous bins, GBT_HIST_ROTATED forces the
 * rotated-feature kernel (features of at most 256 bins; others fall back to
 * the plain one).  GBT_E_INVALID for another value. */
#define GBT_HIST_AUTO 0
#define GBT_HIST_PLAIN 1
#define GBT_HIST_ROTATED 2
gbt_status gbt_ctx_set_hist_kernel(gbt_ctx *ctx, int32_t choice);

/* How the compaction of Alg. 7 (Sec. 3.4) reads pages held in pinned host
 * memory (results are identical): GBT_COMPACT_STREAM copies every page over
 * the host link in chunks and compacts each chunk on the device;
 * GBT_COMPACT_GATHER has the compaction kernel read only the kept rows
 * straight from the pinned pages (device-mapped host memory), so about R of
 * the n rows cross the link; GBT_COMPACT_AUTO gathers when at most half of
 * the rows are kept.  Device-resident pages are read in place either way,
 * and disk pages always stream.
 * GBT_E_INVALID for another value. */
#define GBT_COMPACT_AUTO 0
#define GBT_COMPACT_STREAM 1
#define GBT_COMPACT_GATHER 2
gbt_status gbt_ctx_set_compaction(gbt_ctx *ctx, int32_t mode);

/* Rows per chunk when pages held in pinned host memory or on disk are
 * streamed through the device (Sec. 3.3-3.4: pages are processed in
 * batches; Alg. 7's compaction and the margin update stream them): each
 * chunk is copied (or read from its file, then copied) into one of two
 * device staging buffers of this many rows on the side stream while the
 * previous chunk is processed.  0 restores the default 2^22; results do not
 * depend on the value.  GBT_E_INVALID for rows < 0 or > 2^30. */
gbt_status gbt_ctx_set_stream_chunk_rows(gbt_ctx *ctx, int64_t rows);

/* ---- quantile cuts and ELLPACK pages: Sec. 2.2, Sec. 3.1 (Alg. 2, 3),
 * Sec. 3.2 (Alg. 4, 5) ------------------------------------------------------
 * Cuts are exact quantiles of a sketch sample: for a feature with sorted
 * non-missing sketch values s_0..s_{N-1}, candidate k (1..max_bin-1) is
 * s[ceil(k*N/max_bin)-1]; duplicates and values >= s_{N-1} are dropped;
 * bin(x) = #{cuts < x}.  gbt_quantize is the one-shot form; the incremental
 * form takes batches (Alg. 3 sketch, then Alg. 5 pages):
 *   begin -> sketch_batch* (every batch, in row order) -> finalize_cuts ->
 *   encode_batch* (every batch again, same order) -> end.
 * n_rows_total fixes the sketch stride.
 * sketch_summary = S > 0 selects Alg. 3's merged sketch instead: each
 * sketch_batch call is one batch (gbt_quantize makes one batch of its
 * input); the batch's sample values of every feature, sorted on the device,
 * become a summary -- a list of distinct values v_1 < ... < v_k, each with a
 * count c_i of the values <= v_i: the batch's distinct values with their
 * exact counts when there are at most S, else the values at ranks
 * ceil(tN/S), t = 1..S -- which is merged into the running summary (every
 * value of either, counted c_A(v) + c_B(v) with c_X(v) the count of X's last
 * entry <= v) and pruned back to S entries (entry min{i : c_i >= ceil(tN/S)}
 * for t = 1..S).  The cuts are the exact rule applied to the final summary
 * (candidate k: the value of min{i : c_i >= ceil(kN/max_bin)}), so they equal
 * the exact cuts whenever no summary exceeds S entries.  The device holds one
 * batch's sample keys and 5 * n_cols * S summary entries of 12 bytes, not
 * the whole sample.  page_home DISK writes each page to
 * a file of its own under page_dir (Sec. 3.2: pages on disk), created
 * exclusively and unlinked at once, so the files vanish with the matrix or
 * the process; each tree then reads the pages back through pinned staging
 * buffers, as it streams pinned pages (GBT_E_INVALID without page_dir,
 * GBT_E_IO when a file cannot be created, written or read).  page_home
 * PINNED_HOST keeps pages
 * in page-locked host memory for streaming. */
gbt_status gbt_quantize(gbt_ctx *ctx, const gbt_input *in, const gbt_quant_params *p,
                        gbt_matrix **out);
gbt_status gbt_quantize_begin(gbt_ctx *ctx, const gbt_quant_params *p, int32_t n_cols,
                              int64_t n_rows_total, int32_t input_kind, gbt_quantizer **out);
gbt_status gbt_quantize_sketch_batch(gbt_quantizer *q, const gbt_input *batch);
gbt_status gbt_quantize_finalize_cuts(gbt_quantizer *q);
gbt_status gbt_quantize_encode_batch(gbt_quantizer *q, const gbt_input *batch);
gbt_status gbt_quantize_end(gbt_quantizer *q, gbt_matrix **out); /* frees q */
gbt_status gbt_quantizer_free(gbt_quantizer *q);

gbt_status gbt_matrix_info_get(const gbt_matrix *m, gbt_matrix_info *info);
/* Host copies of the cuts: cut_ptr_h[n_cols+1], cut_values_h[cut_ptr_h[n_cols]]. */
gbt_status gbt_matrix_get_cuts(const gbt_matrix *m, int32_t *cut_ptr_h, float *cut_values_h);
/* Copy page `page` (page_rows[page]*row_words words) to dst (host or device). */
gbt_status gbt_matrix_copy_page(const gbt_matrix *m, int32_t page, void *dst, int64_t dst_words);
gbt_status gbt_matrix_page_rows(const gbt_matrix *m, int32_t page, int64_t *row0, int64_t *rows);
gbt_status gbt_matrix_free(gbt_matrix *m);

/* ---- gradients: Eq. 4-5 ---------------------------------------------------
 * gpair_d[2i], gpair_d[2i+1] = (float) g_i, h_i computed in double:
 *   logistic: s = 1/(1+exp(-z)), g = s - y, h = max(s(1-s), 1e-16)
 *   squared : g = z - y, h = 1
 * times weight_d[i] when weight_d is not NULL. */
gbt_status gbt_gradients(gbt_ctx *ctx, int32_t loss, const float *margin_d, const float *label_d,
                         const float *weight_d, int64_t n, float *gpair_d);

/* ---- sampling and compaction: Sec. 2.4 Eq. 9, Sec. 3.4 Alg. 7 -------------
 * Minimal variance sampling of the n rows of `data` with probability
 * proportional to sqrt(g^2 + mvs_lambda h^2), then compaction of the kept
 * rows (ascending) into one device page, reweighting by the inverse
 * inclusion probability, and exact fixed-point conversion of the reweighted
 * pairs.  Integer reading:
 *   a_i = rint(r_i 2^e), e = 62 - E - ceil(log2 n), max r < 2^E
 *   K = max(1, rint(f n)); T* = least T >= 1 with
 *       sum_{a_i<T} a_i <= (K - #{a_i >= T}) T
 *   keep iff a_i >= T* or hi64(U_i T*) < a_i, U_i = word (i mod 4) of
 *       Philox4x64-10(counter (i div 4, iteration, 0, 0), key (seed, 0))
 *   w_i = 1 if a_i >= T* else T* / a_i;  (g', h') = (g w_i, h w_i)
 *   q = rint((g', h') 2^(e_g, e_h)), e = 62 - E - ceil(log2 R)
 * Sec. 2.3's other samplers (sp->sampler), with the same draws U_i, p < 1
 * compared as U_i < floor(p 2^64) (p = 1 keeps):
 *   GBT_SAMPLE_SGB : keep iff U_i < floor(f 2^64); w_i = 1
 *   GBT_SAMPLE_GOSS: keys k_i = rint(|g_i| 2^e) (the keys above with
 *       mvs_lambda = 0), A = rint(a n), a = sp->goss_a, b = f - a > 0;
 *       t = the A-th largest key (none when A = 0); keep iff k_i >= t or
 *       U_i < floor(p 2^64), p = b / (1 - a); w_i = 1 if k_i >= t else
 *       (1 - a) / b
 * gpair_d (n pairs) may be NULL for pinned-host data: gradients are then
 * recomputed from margin_d/label_d with sp->loss while pages stream.
 * f = 1 keeps every row without copying (is_alias) when the data is one
 * device page. */
gbt_status gbt_sample(gbt_ctx *ctx, const gbt_matrix *data, const float *gpair_d,
                      const float *margin_d, const float *label_d, const gbt_sample_params *sp,
                      gbt_sampled **out);
gbt_status gbt_sampled_info_get(const gbt_sampled *s, gbt_sampled_info *info);
gbt_status gbt_sampled_free(gbt_sampled *s);

/* ---- Alg. 1 BuildHistograms ------------------------------------------------
 * For each build segment: hist_d[slot][off_j + b] += (q_g, q_h) of the rows
 * rows_d[begin..end) (row ids of `page`, NULL = identity) whose symbol for
 * feature j is bin b; missing values add nothing.  hist_d is int64
 * [slots][total_bins][2] and the built slots are overwritten.  Then for each
 * sub entry: hist_d[target] = parent_hist_d[parent] - hist_d[built] (the
 * sibling of a built child), exact in integers.  `page` is a device page of
 * the matrix geometry of `layout` (page_d rows of row_words words), as
 * gbt_quantize writes it, 16-byte aligned (else GBT_E_INVALID).  Symbols
 * outside a feature's bin range (only in a page not written by this library)
 * add nothing.  GBT_E_UNSUPPORTED when a feature has more bins than one
 * histogram group holds (2560 for dense pages, 10176 for sparse ones). */
gbt_status gbt_build_hist(gbt_ctx *ctx, const gbt_matrix *layout, const uint32_t *page_d,
                          const int64_t *gpair_fx_d, const int32_t *rows_d, const gbt_seg *build_h,
                          int32_t n_build, const gbt_sub *sub_h, int32_t n_sub,
                          const int64_t *parent_hist_d, int64_t *hist_d);

/* ---- gbt_build_hist without allocation ------------------------------------
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same
 * arguments and results as gbt_build_hist, with its partial histograms and
 * work plan in a static device array of 64 MiB that every GPU the library
 * runs on holds until the process ends (its address on each device is
 * resolved by gbt_ctx_create).  The call allocates no device memory and
 * records no timing events; it may cut a node's rows into fewer, longer
 * chunks than gbt_build_hist so that they fit (the histograms are the
 * same), and returns GBT_E_INVALID when even one chunk per non-empty node
 * does not fit (about 64 MiB / (total_bins * 16) nodes).  All calls on one
 * GPU share its array: calls that overlap on a GPU (from several threads,
 * contexts or streams) race and give wrong histograms; the call
 * synchronizes its stream before returning, so calls made one after the
 * other are safe. */
gbt_status gbt_build_hist_noalloc(gbt_ctx *ctx, const gbt_matrix *layout, const uint32_t *page_d,
                                  const int64_t *gpair_fx_d, const int32_t *rows_d,
                                  const gbt_seg *build_h, int32_t n_build, const gbt_sub *sub_h,
                                  int32_t n_sub, const int64_t *parent_hist_d, int64_t *hist_d);

/* ---- Alg. 1 EvaluateSplit with Eq. 8 ---------------------------------------
 * For node k: histogram hist_d[node_slot_d[k]], node sum node_sum_d[2k..2k+1]
 * (every array on the device; node_slot_d[k] must name a slot of hist_d).
 * Every feature with >= 2 bins, every s in 1..B_j-1, missing right then
 * left: Q_L = sum_{b<s} H (+ missing sums), Q_R = node - Q_L; valid when
 * H_L, H_R >= min_child_weight; gain = 0.5((G_L^2/(H_L+l) + G_R^2/(H_R+l))
 * - G^2/(H+l)) - gamma in double; the best is the highest gain, ties to the
 * lower feature, lower s, missing right.  out_d[k] receives it, with the
 * split's threshold from the cuts of `layout`.  Enqueued on the context
 * stream without waiting for it (no host round trip): out_d is ready in
 * stream order. */
gbt_status gbt_eval_splits(gbt_ctx *ctx, const gbt_matrix *layout, const int64_t *hist_d,
                           const int64_t *node_sum_d, const int32_t *node_slot_d, int32_t n_nodes,
                           const gbt_train_params *tp, int32_t exp_g, int32_t exp_h,
                           gbt_split *out_d);

/* ---- Alg. 1 RepartitionInstances -------------------------------------------
 * For node k with segment seg_d[k] of rows_d (segments disjoint) and split
 * split_d[k]: when valid, a stable partition of the segment into
 * [left | right] where a row goes left iff its bin for the split feature is
 * < split_bin, or it is missing and default_left, and position_d[row]
 * receives child_d[2k] or child_d[2k+1]; a node that does not split keeps
 * its rows in place.  seg_out_d[2k], seg_out_d[2k+1] receive the child
 * segments {child_d[2k], begin, begin + n_left}, {child_d[2k+1],
 * begin + n_left, end} (the whole segment left when the node does not
 * split).  Every array is on the device (rows_d, rows_tmp_d n_rows entries,
 * 16-byte aligned; rows_d values are rows of page_d; position_d indexed by
 * those rows); rows_tmp_d is scratch.  Enqueued on the context stream
 * without waiting for it: results are ready in stream order.  Malformed
 * entries cannot be reported before the work runs: a segment outside
 * [0, n_rows] is clamped into it, a split feature outside [0, m) does not
 * split, and when status_d (device, may be NULL) is given *status_d
 * receives the number of such nodes plus the number of rows that two
 * segments claim (then the order of those segments' rows is unspecified). */
gbt_status gbt_partition(gbt_ctx *ctx, const gbt_matrix *layout, const uint32_t *page_d,
                         const gbt_split *split_d, const gbt_seg *seg_d, const int32_t *child_d,
                         int32_t n_nodes, int32_t *rows_d, int32_t *rows_tmp_d, int64_t n_rows,
                         int32_t *position_d, gbt_seg *seg_out_d, int32_t *status_d);

/* ---- Eq. 6 leaves and the Eq. 1 margin update -------------------------------
 * Leaves of `tree` (flags LEAF) get leaf_value = (float)((-G/(H+lambda))*eta)
 * from their fixed-point sums; then margin_d[i] += leaf(tree, row i) for the
 * n rows of `data`.  The training rows whose leaf is known take it from
 * their positions: entry i < n_pos names row rows_d[i] of `data` (i when
 * rows_d is NULL; distinct rows, as gbt_sampled_info's rows_d) and its node
 * position_d[i] (as gbt_partition leaves it after the last level); the
 * other rows are traversed by their binned symbols.  Entries whose position
 * is not a leaf of the tree, or whose row is out of range or repeated, are
 * counted and their rows traversed instead: the margins are right, and the
 * call returns GBT_E_INVALID with the count.  Synchronizes the context
 * stream (the tree's leaf values are written back to `tree`). */
gbt_status gbt_update_leaves(gbt_ctx *ctx, gbt_tree *tree, const gbt_train_params *tp,
                             const gbt_matrix *data, const int32_t *rows_d, const int32_t *position_d,
                             int64_t n_pos, float *margin_d);

/* ---- one boosting iteration: Alg. 7 then Alg. 1 -----------------------------
 * Gradients, sampling (f < 1) with compaction into one device page, the
 * level-wise tree (histograms with the sibling subtraction, splits,
 * partitions), leaves and the margin update of all rows.  Pinned-host
 * matrices stream their pages.  tree->nodes must hold 2^(max_depth+1)-1
 * nodes. */
gbt_status gbt_train_tree(gbt_ctx *ctx, const gbt_matrix *data, const float *label_d,
                          float *margin_d, const gbt_train_params *p, gbt_tree *tree,
                          gbt_tree_stats *stats);

/* ---- n_trees boosting iterations: Alg. 1's loop over trees ------------------
 * The same as n_trees calls of gbt_train_tree with p->iteration,
 * p->iteration + 1, ... (the same trees, margins and stats, bit for bit):
 * trees[t] (each holding 2^(max_depth+1)-1 nodes) and stats[t] (stats may
 * be NULL) receive tree t, and margin_d holds the margins after the last
 * tree.  Each tree is queued on the context stream without waiting for the
 * tree before it (no host round trip separates them); the trees' results
 * are read from a ring of pinned host memory the context keeps (64 trees'
 * results, at most 64 MiB, or two when one exceeds 32 MiB) as it fills,
 * and the rest when the stream has drained.  The call returns with the
 * stream synchronized.  n_trees = 0 does nothing.  On an error the trees
 * from the failing one on, and the margins, are undefined. */
gbt_status gbt_train_trees(gbt_ctx *ctx, const gbt_matrix *data, const float *label_d,
                           float *margin_d, const gbt_train_params *p, int32_t n_trees,
                           gbt_tree *trees, gbt_tree_stats *stats);

/* ---- Alg. 6: the naive out-of-core tree construction (Sec. 3.3) ------------
 * A measured negative baseline, not the path to use: every row trains
 * (p->f must be 1) and each level streams every page of `data` once,
 * moving each row to its node and building the histograms of all of the
 * level's nodes from each chunk (no sibling subtraction, since no page stays
 * on the device); one last pass moves the rows to the leaves, whose ids
 * give the margin update.  Tree, margins and stats as gbt_train_tree's with
 * f = 1 (the same tree, bit for bit); p->max_depth <= 11.  Holds a node id
 * (4 bytes) and the fixed-point pair (16 bytes) of every row on the device. */
gbt_status gbt_train_tree_naive(gbt_ctx *ctx, const gbt_matrix *data, const float *label_d,
                                float *margin_d, const gbt_train_params *params, gbt_tree *tree_out,
                                gbt_tree_stats *stats);

/* ---- MVS lambda estimated from the data: Sec. 2.4 ---------------------------
 * *lambda_out = w0^2 with w0 = -G/H the initial leaf value, read as the
 * unregularized Newton step of all n rows at margin_d (length n, device):
 * G and H are the exact integer sums of the rows' gradients (Eq. 4-5, loss
 * as in gbt_gradients) in their fixed point over the n rows (the
 * representation the histograms use), scaled back to double; 0 when H or n
 * is 0.  Pass the value as mvs_lambda of later iterations.  Synchronizes
 * the context stream. */
gbt_status gbt_mvs_lambda_estimate(gbt_ctx *ctx, int32_t loss, const float *margin_d,
                                   const float *label_d, int64_t n, double *lambda_out);

/* ---- Eq. 1 prediction -------------------------------------------------------
 * margin_out_d[i] = base_margin + sum_t leaf(tree t, row i), in float, tree
 * order.  Exactly one of raw (rows traverse by x <= threshold, missing by
 * default_left; must be device resident) or binned (symbols) is given. */
gbt_status gbt_predict(gbt_ctx *ctx, const gbt_tree *trees, int32_t n_trees,
                       const gbt_input *raw, const gbt_matrix *binned, float base_margin,
                       float *margin_out_d);

#ifdef __cplusplus
}
#endif

#endif /* GBT_H */
