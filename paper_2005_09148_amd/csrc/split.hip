// split.hip -- Alg. 1 EvaluateSplit with the loss reduction of Eq. 8, and
// Alg. 1 RepartitionInstances (stable, scan based).
//
// Evaluation: one wavefront per (node, feature).  Each lane holds four
// consecutive bins; an int64 wavefront prefix scan gives the left sums of
// every cut s, the missing sums come from node sum minus the feature's bin
// total, and every (s, direction) gain is computed in double exactly as
// 0.5*((G_L^2/(H_L+l) + G_R^2/(H_R+l)) - G^2/(H+l)) - gamma.  The best is
// the highest gain; ties go to the lower feature, then the lower s, then
// missing-right.
//
// Partition: per training slot a left flag from the row's symbol of the
// split feature, a device-wide exclusive scan of the flags, and a scatter
// that writes [left | right] of every splitting segment in input order.
#include "split_impl.h"
#include "plan_impl.h"
#include "wave_impl.h"

#include <cstring>

namespace gbt {

constexpr int kEvalThreads = 256;
constexpr int kFeatPerBlock = 4;

struct Cand {
    double gain;
    int32_t order;  // s*2 + dir within a feature, or feature index across features
    int32_t valid;
    long long lg, lh;
};

__device__ inline bool better(const Cand &a, const Cand &b)
{
    // a strictly preferred over b
    if (!a.valid) return false;
    if (!b.valid) return true;
    if (a.gain > b.gain) return true;
    if (a.gain < b.gain) return false;
    return a.order < b.order;
}

__device__ inline double fx(long long Q, int32_t e) { return ldexp((double)Q, -e); }

// The split's raw-value form: bins < split_bin hold the values <= the cut
// below bin split_bin.
__device__ inline float split_threshold(const SplitCuts &c, int32_t feature, int32_t split_bin)
{
    return c.values[c.ptr[feature] + split_bin - 1];
}

// Eq. 8: 0.5*((G_L^2/(H_L+lambda) + G_R^2/(H_R+lambda)) - c) - gamma, with
// the parent's term c = G^2/(H+lambda) computed once per node.
__device__ inline double eq8_gain_c(double GL, double HL, double GR, double HR, double c, double lambda,
                                    double gamma)
{
    double a = (GL * GL) / (HL + lambda);
    double b = (GR * GR) / (HR + lambda);
    return 0.5 * ((a + b) - c) - gamma;
}

// A lane's kN candidates of one feature: every gain is computed before any
// is compared (the divisions of different candidates overlap instead of
// waiting on each other's branches), then the candidates are taken in
// (s, dir) order exactly as a loop that skips the inadmissible ones would.
// lg/lh: left sums; s: the cut (left = bins < s) of candidate k / 2.
template <int kN>
__device__ inline void pick_candidates(const long long *lg, const long long *lh, const int32_t *s, int32_t B,
                                       long long Qg, long long Qh, double c, const EvalParams &ep, Cand &best)
{
    double gain[kN];
    bool ok[kN];
#pragma unroll
    for (int k = 0; k < kN; ++k) {
        const double GL = fx(lg[k], ep.e_g), HL = fx(lh[k], ep.e_h);
        const double GR = fx(Qg - lg[k], ep.e_g), HR = fx(Qh - lh[k], ep.e_h);
        gain[k] = eq8_gain_c(GL, HL, GR, HR, c, ep.lambda, ep.gamma);
        // no short circuit: the gain is needed whatever the other tests say,
        // so its division is not moved under a branch of its own
        ok[k] = (s[k / 2] <= B - 1) & (HL >= ep.mcw) & (HR >= ep.mcw) & (gain[k] == gain[k]);
    }
    // better() as selects, without branches
#pragma unroll
    for (int k = 0; k < kN; ++k) {
        const int32_t order = s[k / 2] * 2 + (k & 1);
        const bool take = ok[k] & (!best.valid | (gain[k] > best.gain) |
                                   ((gain[k] == best.gain) & (order < best.order)));
        best.gain = take ? gain[k] : best.gain;
        best.order = take ? order : best.order;
        best.valid = take ? 1 : best.valid;
        best.lg = take ? lg[k] : best.lg;
        best.lh = take ? lh[k] : best.lh;
    }
}

// The best candidate of the wavefront (every lane receives it): the highest
// gain among valid lanes, then the lowest order; one max reduction, one min
// reduction and a broadcast from the winning lane.
__device__ inline Cand wave_best(Cand x)
{
    const unsigned long long any = __ballot(x.valid != 0);
    Cand r;
    r.valid = 0;
    r.gain = 0.0;
    r.order = 0;
    r.lg = r.lh = 0;
    if (!any) return r;
    const double m = wave_max_f64(x.valid ? x.gain : -__builtin_inf());
    const bool cand = x.valid && x.gain == m;
    const int32_t o = wave_min<int32_t>(cand ? x.order : 0x7fffffff);
    const unsigned long long win = __ballot(cand && x.order == o);
    const int wl = __ffsll((long long)win) - 1;
    r.valid = 1;
    r.gain = wave_read(x.gain, wl);  // the winner's own bits (+0 and -0 compare equal)
    r.order = o;
    r.lg = wave_read(x.lg, wl);
    r.lh = wave_read(x.lh, wl);
    return r;
}

__device__ inline long long wave_sum(long long v) { return wave_total(v); }

// Best split of one feature for one node, evaluated by one wavefront.  The
// result (valid in every lane) carries order = s*2 + dir.
// The gains of the four cuts after this lane's bins of one 256-bin chunk:
// pg, ph enter as the sums of all bins before the lane's first bin.
__device__ inline void eval_chunk(const longlong2 v[4], int32_t base, int32_t B, long long pg, long long ph,
                                  long long Qg, long long Qh, long long mg, long long mh, double c,
                                  const EvalParams &ep, Cand &best)
{
    const int lane = threadIdx.x & 63;
    long long lg[8], lh[8];
    int32_t s[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        pg += v[t].x;
        ph += v[t].y;
        s[t] = base + lane * 4 + t + 1;  // left = bins < s
#pragma unroll
        for (int dir = 0; dir < 2; ++dir) {
            lg[2 * t + dir] = pg + (dir ? mg : 0);
            lh[2 * t + dir] = ph + (dir ? mh : 0);
        }
    }
    pick_candidates<8>(lg, lh, s, B, Qg, Qh, c, ep, best);
}

// Inclusive wavefront scan of a pair of int64 values.
__device__ inline void wave_scan2(long long &xg, long long &xh)
{
    xg = wave_incl_sum(xg);
    xh = wave_incl_sum(xh);
}

// Best split of one feature for one node, evaluated by one wavefront.  The
// result (valid in every lane) carries order = s*2 + dir.
__device__ Cand eval_feature(const longlong2 *__restrict__ hj, int32_t B, long long Qg, long long Qh,
                             const EvalParams &ep)
{
    const int lane = threadIdx.x & 63;
    Cand best;
    best.valid = 0;
    best.gain = 0.0;
    best.order = 0;
    best.lg = best.lh = 0;
    const double G = fx(Qg, ep.e_g), H = fx(Qh, ep.e_h);
    const double c = (G * G) / (H + ep.lambda);
    if (B <= 256) {
        // one chunk: the scan's last lane holds the feature's bin totals
        longlong2 v[4];
        long long sg = 0, sh = 0;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const int32_t b = lane * 4 + t;
            v[t] = b < B ? hj[b] : make_longlong2(0, 0);
            sg += v[t].x;
            sh += v[t].y;
        }
        long long xg = sg, xh = sh;
        wave_scan2(xg, xh);
        const long long tg = wave_read(xg, 63), th = wave_read(xh, 63);
        eval_chunk(v, 0, B, xg - sg, xh - sh, Qg, Qh, Qg - tg, Qh - th, c, ep, best);
        return wave_best(best);
    }
    // totals over the feature's bins -> missing sums
    long long tg = 0, th = 0;
    for (int32_t b = lane; b < B; b += 64) {
        longlong2 v = hj[b];
        tg += v.x;
        th += v.y;
    }
    tg = wave_sum(tg);
    th = wave_sum(th);
    const long long mg = Qg - tg, mh = Qh - th;
    long long carry_g = 0, carry_h = 0;
    for (int32_t base = 0; base < B; base += 256) {
        longlong2 v[4];
        long long sg = 0, sh = 0;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const int32_t b = base + lane * 4 + t;
            v[t] = b < B ? hj[b] : make_longlong2(0, 0);
            sg += v[t].x;
            sh += v[t].y;
        }
        long long xg = sg, xh = sh;
        wave_scan2(xg, xh);
        eval_chunk(v, base, B, carry_g + xg - sg, carry_h + xh - sh, Qg, Qh, mg, mh, c, ep, best);
        carry_g += wave_read(xg, 63);
        carry_h += wave_read(xh, 63);
    }
    return wave_best(best);
}

// The best of node k's per-feature-block candidates as a gbt_split; with
// `decide` given, a node whose best valid gain is > 0 is also marked as
// split in the tree driver's node table (depth < max_depth is the caller's).
__device__ inline void reduce_node(const EvalCand *cand, int32_t n_fblocks, const EvalNode &node, int32_t k,
                                   gbt_split *__restrict__ out, DevNode *__restrict__ decide, SplitCuts cuts)
{
    EvalCand b;
    b.valid = 0;
    for (int32_t f = 0; f < n_fblocks; ++f) {
        const EvalCand &o = cand[(int64_t)k * n_fblocks + f];
        if (!o.valid) continue;
        if (!b.valid || o.gain > b.gain) b = o;
    }
    gbt_split s;
    s.valid = b.valid;
    s.gain = b.valid ? b.gain : 0.0;
    s.feature = b.valid ? b.feature : -1;
    s.split_bin = b.valid ? b.split_bin : -1;
    s.default_left = b.valid ? b.default_left : 0;
    s.left_g = b.valid ? b.lg : 0;
    s.left_h = b.valid ? b.lh : 0;
    s.right_g = b.valid ? node.sum_g - b.lg : 0;
    s.right_h = b.valid ? node.sum_h - b.lh : 0;
    s.threshold = b.valid ? split_threshold(cuts, b.feature, b.split_bin) : 0.0f;
    s.pad0 = 0;
    out[k] = s;
    if (decide && s.valid && s.gain > 0.0) {
        DevNode &d = decide[node.heap];
        d.split = 1;
        d.feature = s.feature;
        d.split_bin = s.split_bin;
        d.default_left = s.default_left;
        d.gain = s.gain;
        d.left_g = s.left_g;
        d.left_h = s.left_h;
        d.right_g = s.right_g;
        d.right_h = s.right_h;
    }
}

__global__ void k_eval_reduce(const EvalCand *__restrict__ cand, int32_t n_fblocks,
                              const EvalNode *__restrict__ nodes, int32_t n_nodes,
                              const int32_t *__restrict__ n_nodes_d, gbt_split *__restrict__ out,
                              DevNode *__restrict__ decide, SplitCuts cuts)
{
    int32_t k = blockIdx.x * blockDim.x + threadIdx.x;
    if (k >= n_nodes || (n_nodes_d && k >= *n_nodes_d)) return;
    reduce_node(cand, n_fblocks, nodes[k], k, out, decide, cuts);
}

__global__ void __launch_bounds__(kEvalThreads)
    k_eval(const longlong2 *__restrict__ hist, int64_t total_bins, const EvalNode *__restrict__ nodes,
           const int32_t *__restrict__ n_nodes_d, const int32_t *__restrict__ bin_ptr, int32_t m,
           EvalParams ep, EvalCand *__restrict__ out)
{
    __shared__ EvalCand wbest[kEvalThreads / 64];
    if (n_nodes_d && (int32_t)blockIdx.y >= *n_nodes_d) return;
    if (ep.e_dev) {
        ep.e_g = ep.e_dev[0];
        ep.e_h = ep.e_dev[1];
    }
    const EvalNode nd = nodes[blockIdx.y];
    const int wid = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const longlong2 *h = hist + (int64_t)nd.slot * total_bins;
    EvalCand mine;
    mine.valid = 0;
    mine.gain = 0.0;
    mine.feature = -1;
    mine.split_bin = -1;
    mine.default_left = 0;
    mine.lg = mine.lh = 0;
    const int32_t f_end = min(m, (int32_t)(blockIdx.x + 1) * kFeatPerBlock);
    for (int32_t j = blockIdx.x * kFeatPerBlock + wid; j < f_end; j += kEvalThreads / 64) {
        const int32_t b0 = bin_ptr[j], B = bin_ptr[j + 1] - b0;
        if (B < 2) continue;
        Cand c = eval_feature(h + b0, B, nd.sum_g, nd.sum_h, ep);
        // features visited in ascending order: keep the first of equal gains
        if (c.valid && (!mine.valid || c.gain > mine.gain)) {
            mine.valid = 1;
            mine.gain = c.gain;
            mine.feature = j;
            mine.split_bin = c.order >> 1;
            mine.default_left = c.order & 1;
            mine.lg = c.lg;
            mine.lh = c.lh;
        }
    }
    if (lane == 0) wbest[wid] = mine;
    __syncthreads();
    if (threadIdx.x == 0) {
        EvalCand b = wbest[0];
        for (int w = 1; w < kEvalThreads / 64; ++w) {
            const EvalCand &o = wbest[w];
            if (!o.valid) continue;
            if (!b.valid || o.gain > b.gain || (o.gain == b.gain && o.feature < b.feature)) b = o;
        }
        out[(int64_t)blockIdx.y * gridDim.x + blockIdx.x] = b;
    }
}

// ------------------------------------------------------------ reduce + evaluate
// One block per (feature, reduce item): 4 waves cover the feature's bins 64
// at a time, and kSub such wave sets take every kSub-th partial; the built
// node's and the sibling's bins go to hist (unless hist is NULL: the level's
// histograms are parents of no later level) and to LDS, then wave 0
// evaluates the built node and wave 1 the sibling on the LDS copy.  Levels
// of few nodes and many partials per node use kSub = 4 (1024 threads);
// levels of many nodes use kSub = 1 (256 threads), so that more blocks are
// resident while two waves of each evaluate.
template <int kSub>
__global__ void __launch_bounds__(256 * kSub)
    k_reduce_eval(const longlong2 *__restrict__ partials, const HistReduce *__restrict__ red,
                  const int32_t *__restrict__ n_red_d, const longlong2 *__restrict__ parent,
                  longlong2 *__restrict__ hist, int64_t total_bins, const int32_t *__restrict__ bin_ptr,
                  int32_t m, const EvalNode *__restrict__ ev, EvalParams ep, EvalCand *__restrict__ cand)
{
    if (n_red_d && (int32_t)blockIdx.y >= *n_red_d) return;
    __shared__ longlong2 hb[256], hs[256];
    __shared__ long long sg[kSub][256], sh[kSub][256];
    const HistReduce rd = red[blockIdx.y];
    const int32_t f = blockIdx.x;
    const int32_t b0 = bin_ptr[f], B = bin_ptr[f + 1] - b0;
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    const int sub = wid >> 2;                 // partial subset
    const int32_t b = (wid & 3) * 64 + lane;  // bin of the feature (B <= 256)
    const bool sib = rd.sub_target >= 0;
    long long g = 0, h = 0;
    if (b < B) {
        const longlong2 *src = partials + (int64_t)rd.part0 * total_bins + b0 + b;
        int32_t k = sub;
        // eight loads in flight per thread
        for (; k + 7 * kSub < rd.nparts; k += 8 * kSub) {
            longlong2 v[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) v[j] = src[(int64_t)(k + j * kSub) * total_bins];
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                g += v[j].x;
                h += v[j].y;
            }
        }
        for (; k < rd.nparts; k += kSub) {
            const longlong2 v = src[(int64_t)k * total_bins];
            g += v.x;
            h += v.y;
        }
    }
    sg[sub][b] = g;
    sh[sub][b] = h;
    __syncthreads();
    if (sub == 0 && b < B) {
        for (int t = 1; t < kSub; ++t) {
            g += sg[t][b];
            h += sh[t][b];
        }
        const longlong2 bv = make_longlong2(g, h);
        if (hist) hist[(int64_t)rd.slot * total_bins + b0 + b] = bv;
        hb[b] = bv;
        if (sib) {
            const longlong2 pv = parent[(int64_t)rd.sub_parent * total_bins + b0 + b];
            const longlong2 sv = make_longlong2(pv.x - g, pv.y - h);
            if (hist) hist[(int64_t)rd.sub_target * total_bins + b0 + b] = sv;
            hs[b] = sv;
        }
    }
    __syncthreads();
    if (wid > (sib ? 1 : 0)) return;
    const int32_t slot = wid == 0 ? rd.slot : rd.sub_target;
    if (ep.e_dev) {
        ep.e_g = ep.e_dev[0];
        ep.e_h = ep.e_dev[1];
    }
    EvalCand o;
    o.valid = 0;
    o.gain = 0.0;
    o.feature = f;
    o.split_bin = -1;
    o.default_left = 0;
    o.lg = o.lh = 0;
    if (B >= 2) {
        const EvalNode nd = ev[slot];
        const Cand cb = eval_feature(wid == 0 ? hb : hs, B, nd.sum_g, nd.sum_h, ep);
        if (cb.valid) {
            o.valid = 1;
            o.gain = cb.gain;
            o.split_bin = cb.order >> 1;
            o.default_left = cb.order & 1;
            o.lg = cb.lg;
            o.lh = cb.lh;
        }
    }
    if (lane == 0) cand[(int64_t)slot * m + f] = o;
}

// Best split of one feature of at most 64 kBL bins for one node, held in
// registers: lane l's t-th value is bin t * 64 + l (zeros past B).  The same
// cuts, gains and choice as eval_feature.
template <int kBL>
__device__ Cand eval_feature_regs(const long long *g, const long long *h, int32_t B, long long Qg, long long Qh,
                                  const EvalParams &ep)
{
    const int lane = threadIdx.x & 63;
    Cand best;
    best.valid = 0;
    best.gain = 0.0;
    best.order = 0;
    best.lg = best.lh = 0;
    const double G = fx(Qg, ep.e_g), H = fx(Qh, ep.e_h);
    // inclusive prefix sums in bin order: chunk by chunk, each carried by
    // the totals of the chunks before it; the last carry is the total
    long long pgs[kBL], phs[kBL];
    long long cg = 0, ch = 0;
#pragma unroll
    for (int t = 0; t < kBL; ++t) {
        long long xg = g[t], xh = h[t];
        wave_scan2(xg, xh);
        pgs[t] = cg + xg;
        phs[t] = ch + xh;
        cg += wave_read(xg, 63);
        ch += wave_read(xh, 63);
    }
    const long long mg = Qg - cg, mh = Qh - ch;
    long long lg[2 * kBL], lh[2 * kBL];
    int32_t s[kBL];
#pragma unroll
    for (int t = 0; t < kBL; ++t) {
        s[t] = t * 64 + lane + 1;  // left = bins < s
#pragma unroll
        for (int dir = 0; dir < 2; ++dir) {
            lg[2 * t + dir] = pgs[t] + (dir ? mg : 0);
            lh[2 * t + dir] = phs[t] + (dir ? mh : 0);
        }
    }
    pick_candidates<2 * kBL>(lg, lh, s, B, Qg, Qh, (G * G) / (H + ep.lambda), ep, best);
    return wave_best(best);
}

// k_reduce_eval with the histograms in registers: a wave takes 4 / kBL
// features of one node (features of at most 64 kBL bins), lane l bins
// l, l + 64, ...; the parent's and the partials' loads of all of them are
// in flight together.  No LDS and no block barrier.  blockIdx.z = 0 sums the
// built node's partials, writes its histogram and evaluates it; z = 1 does
// the same for its sibling (parent minus the sums), so the two evaluations
// run side by side.
template <int kBL>
__global__ void __launch_bounds__(256)
    k_reduce_eval_regs(const longlong2 *__restrict__ partials, const HistReduce *__restrict__ red,
                       const int32_t *__restrict__ n_red_d, const longlong2 *__restrict__ parent,
                       longlong2 *__restrict__ hist, int64_t total_bins, const int32_t *__restrict__ bin_ptr,
                       int32_t m, const EvalNode *__restrict__ ev, EvalParams ep, EvalCand *__restrict__ cand)
{
    constexpr int kFW = 4 / kBL;  // features per wave
    constexpr int kV = kFW * kBL; // values per lane
    if (n_red_d && (int32_t)blockIdx.y >= *n_red_d) return;
    const int lane = threadIdx.x & 63;
    const int32_t f0 = (int32_t)(blockIdx.x * 4 + (threadIdx.x >> 6)) * kFW;
    if (f0 >= m) return;  // the whole wave
    const HistReduce rd = red[blockIdx.y];
    const bool sib = rd.sub_target >= 0;
    const int which = (int)blockIdx.z;
    if (which == 1 && !sib) return;
    int32_t off[kV];  // bin offset of each value, -1 past its feature's bins
#pragma unroll
    for (int j = 0; j < kFW; ++j) {
        const int32_t f = f0 + j;
        int32_t b0 = 0, B = 0;
        if (f < m) {
            b0 = bin_ptr[f];
            B = bin_ptr[f + 1] - b0;
        }
#pragma unroll
        for (int t = 0; t < kBL; ++t) off[j * kBL + t] = t * 64 + lane < B ? b0 + t * 64 + lane : -1;
    }
    longlong2 pv[kV];
#pragma unroll
    for (int i = 0; i < kV; ++i)
        pv[i] = (which == 1 && off[i] >= 0) ? parent[(int64_t)rd.sub_parent * total_bins + off[i]]
                                            : make_longlong2(0, 0);
    long long g[kV], h[kV];
#pragma unroll
    for (int i = 0; i < kV; ++i) g[i] = h[i] = 0;
    const longlong2 *src = partials + (int64_t)rd.part0 * total_bins;
    int32_t k = 0;
    for (; k + 1 < rd.nparts; k += 2) {
        longlong2 v[2][kV];
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
            for (int i = 0; i < kV; ++i)
                v[u][i] = off[i] >= 0 ? src[(int64_t)(k + u) * total_bins + off[i]] : make_longlong2(0, 0);
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
            for (int i = 0; i < kV; ++i) {
                g[i] += v[u][i].x;
                h[i] += v[u][i].y;
            }
    }
    if (k < rd.nparts) {
#pragma unroll
        for (int i = 0; i < kV; ++i) {
            const longlong2 v = off[i] >= 0 ? src[(int64_t)k * total_bins + off[i]] : make_longlong2(0, 0);
            g[i] += v.x;
            h[i] += v.y;
        }
    }
    // z = 1: the sibling in place of the built node
    if (which == 1) {
#pragma unroll
        for (int i = 0; i < kV; ++i) {
            g[i] = pv[i].x - g[i];
            h[i] = pv[i].y - h[i];
        }
    }
    const int32_t slot = which == 0 ? rd.slot : rd.sub_target;
    if (hist) {
#pragma unroll
        for (int i = 0; i < kV; ++i)
            if (off[i] >= 0) hist[(int64_t)slot * total_bins + off[i]] = make_longlong2(g[i], h[i]);
    }
    if (ep.e_dev) {
        ep.e_g = ep.e_dev[0];
        ep.e_h = ep.e_dev[1];
    }
    {
        const EvalNode nd = ev[slot];
#pragma unroll
        for (int j = 0; j < kFW; ++j) {
            const int32_t f = f0 + j;
            if (f >= m) break;
            const int32_t B = bin_ptr[f + 1] - bin_ptr[f];
            EvalCand o;
            o.valid = 0;
            o.gain = 0.0;
            o.feature = f;
            o.split_bin = -1;
            o.default_left = 0;
            o.lg = o.lh = 0;
            if (B >= 2) {
                const Cand cb = eval_feature_regs<kBL>(g + j * kBL, h + j * kBL, B, nd.sum_g, nd.sum_h, ep);
                if (cb.valid) {
                    o.valid = 1;
                    o.gain = cb.gain;
                    o.split_bin = cb.order >> 1;
                    o.default_left = cb.order & 1;
                    o.lg = cb.lg;
                    o.lh = cb.lh;
                }
            }
            if (lane == 0) cand[(int64_t)slot * m + f] = o;
        }
    }
}

// Each node's best candidate over its features, one wave per node: the
// highest gain, ties to the lowest feature (candidates are in feature order).
__global__ void __launch_bounds__(256)
    k_eval_reduce_wave(const EvalCand *__restrict__ cand, int32_t n_fblocks, const EvalNode *__restrict__ nodes,
                       int32_t n_nodes, const int32_t *__restrict__ n_nodes_d, gbt_split *__restrict__ out,
                       DevNode *__restrict__ decide, SplitCuts cuts)
{
    const int lane = threadIdx.x & 63;
    const int32_t k = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (k >= n_nodes || (n_nodes_d && k >= *n_nodes_d)) return;
    // each lane keeps the best of its features (ascending), then the wave
    // takes the highest gain and, among equal gains, the lowest feature
    int32_t bi = -1;
    double bg = 0.0;
    for (int32_t f = lane; f < n_fblocks; f += 64) {
        const EvalCand &o = cand[(int64_t)k * n_fblocks + f];
        if (o.valid && (bi < 0 || o.gain > bg)) {
            bi = f;
            bg = o.gain;
        }
    }
    const double m = wave_max_f64(bi >= 0 ? bg : -__builtin_inf());
    const int32_t best = wave_min<int32_t>((bi >= 0 && bg == m) ? bi : 0x7fffffff);
    if (lane != 0) return;
    const EvalCand b = best != 0x7fffffff ? cand[(int64_t)k * n_fblocks + best] : EvalCand{0.0, 0, 0, -1, -1, 0, 0};
    const EvalNode node = nodes[k];
    gbt_split sp;
    sp.valid = b.valid;
    sp.gain = b.valid ? b.gain : 0.0;
    sp.feature = b.valid ? b.feature : -1;
    sp.split_bin = b.valid ? b.split_bin : -1;
    sp.default_left = b.valid ? b.default_left : 0;
    sp.left_g = b.valid ? b.lg : 0;
    sp.left_h = b.valid ? b.lh : 0;
    sp.right_g = b.valid ? node.sum_g - b.lg : 0;
    sp.right_h = b.valid ? node.sum_h - b.lh : 0;
    sp.threshold = b.valid ? split_threshold(cuts, b.feature, b.split_bin) : 0.0f;
    sp.pad0 = 0;
    out[k] = sp;
    if (decide && sp.valid && sp.gain > 0.0) {
        DevNode &d = decide[node.heap];
        d.split = 1;
        d.feature = sp.feature;
        d.split_bin = sp.split_bin;
        d.default_left = sp.default_left;
        d.gain = sp.gain;
        d.left_g = sp.left_g;
        d.left_h = sp.left_h;
        d.right_g = sp.right_g;
        d.right_h = sp.right_h;
    }
}

gbt_status reduce_eval_impl(gbt_ctx *c, const gbt_matrix *mx, const int64_t *partials, const HistReduce *red,
                            const int32_t *n_red_d, int32_t max_red, const int64_t *parent, int64_t *hist,
                            const EvalNode *ev, const EvalParams &ep, EvalCand *cand)
{
    if (max_red <= 0) return GBT_OK;
    int32_t max_feature_bins = 0;
    for (int32_t f = 0; f < mx->m; ++f)
        max_feature_bins = std::max(max_feature_bins, mx->bin_ptr_h[f + 1] - mx->bin_ptr_h[f]);
    // features of at most 64 bins, or many (feature, node) pairs: the
    // register form (a wave per 1, 2 or 4 features)
    const int kbl = max_feature_bins <= 64 ? 1 : max_feature_bins <= 128 ? 2 : max_feature_bins <= 256 ? 4 : 0;
    if (kbl == 1 || (kbl > 0 && (int64_t)max_red * mx->m >= 2 * kCUs)) {
        const int fpb = 4 * (4 / kbl);  // features per block
        // z: the built node and, below the root, its sibling
        dim3 gr((unsigned)((mx->m + fpb - 1) / fpb), (unsigned)max_red, parent ? 2u : 1u);
#define GBT_REG_EVAL(BL)                                                                                       \
    k_reduce_eval_regs<BL><<<gr, 256, 0, c->stream>>>((const longlong2 *)partials, red, n_red_d,           \
                                                      (const longlong2 *)parent, (longlong2 *)hist,         \
                                                      mx->total_bins, mx->bin_ptr_d, mx->m, ev, ep, cand)
        if (kbl == 1)
            GBT_REG_EVAL(1);
        else if (kbl == 2)
            GBT_REG_EVAL(2);
        else
            GBT_REG_EVAL(4);
#undef GBT_REG_EVAL
        GBT_LAUNCHED();
        return GBT_OK;
    }
    dim3 grid((unsigned)mx->m, (unsigned)max_red);
    // many (feature, node) blocks: the narrow form keeps more of them resident
    if ((int64_t)max_red * mx->m >= 2 * kCUs)
        k_reduce_eval<1><<<grid, 256, 0, c->stream>>>((const longlong2 *)partials, red, n_red_d,
                                                      (const longlong2 *)parent, (longlong2 *)hist,
                                                      mx->total_bins, mx->bin_ptr_d, mx->m, ev, ep, cand);
    else
        k_reduce_eval<4><<<grid, 1024, 0, c->stream>>>((const longlong2 *)partials, red, n_red_d,
                                                       (const longlong2 *)parent, (longlong2 *)hist,
                                                       mx->total_bins, mx->bin_ptr_d, mx->m, ev, ep, cand);
    GBT_LAUNCHED();
    return GBT_OK;
}

gbt_status eval_reduce_impl(gbt_ctx *c, const gbt_matrix *mx, const EvalCand *cand, int32_t n_fblocks,
                            const EvalNode *nodes_d, int32_t n_nodes, const int32_t *n_nodes_d, gbt_split *out_d,
                            DevNode *decide)
{
    if (n_nodes <= 0) return GBT_OK;
    k_eval_reduce_wave<<<(n_nodes + 3) / 4, 256, 0, c->stream>>>(cand, n_fblocks, nodes_d, n_nodes, n_nodes_d,
                                                                 out_d, decide, cuts_of(mx));
    GBT_LAUNCHED();
    return GBT_OK;
}

gbt_status eval_impl(gbt_ctx *c, const gbt_matrix *mx, const int64_t *hist, const EvalNode *nodes_d,
                     int32_t n_nodes, const EvalParams &ep, gbt_split *out_d, const int32_t *n_nodes_d,
                     DevNode *decide)
{
    if (n_nodes == 0) return GBT_OK;
    int32_t nfb = (mx->m + kFeatPerBlock - 1) / kFeatPerBlock;
    EvalCand *cand;
    GBT_TRY(scratch_t(c, kScrEval, (size_t)n_nodes * nfb, &cand));
    dim3 grid((unsigned)nfb, (unsigned)n_nodes);
    k_eval<<<grid, kEvalThreads, 0, c->stream>>>((const longlong2 *)hist, mx->total_bins, nodes_d, n_nodes_d,
                                                 mx->bin_ptr_d, mx->m, ep, cand);
    GBT_LAUNCHED();
    k_eval_reduce<<<(n_nodes + 127) / 128, 128, 0, c->stream>>>(cand, nfb, nodes_d, n_nodes, n_nodes_d, out_d,
                                                                decide, cuts_of(mx));
    GBT_LAUNCHED();
    return GBT_OK;
}

// ------------------------------------------------------------ partition
// Slots are processed in tiles of 1024, one 256-thread block per tile (small
// blocks keep several tiles in flight on each CU); a thread owns four
// consecutive slots, so its row ids, node ids and flags are one vector load
// each, and the loads of the four slots are issued together.
constexpr int kPartThreads = 256;
constexpr int kPartItems = 4;
constexpr int kPartTile = kPartThreads * kPartItems;  // the scan's tile

// Exclusive sum over a block of kPartThreads; *total receives the block's sum.
__device__ inline int32_t part_block_scan(int32_t v, int32_t *lds16, int32_t *total)
{
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    const int32_t x = wave_incl_sum(v);
    if (lane == 63) lds16[wid] = x;
    __syncthreads();
    int32_t off = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < kPartThreads / 64; ++w) {
        const int32_t t = lds16[w];
        off += w < wid ? t : 0;
        tot += t;
    }
    *total = tot;
    return x - v + off;
}

// The four slots' row ids and node ids (node of slot i: slot_node[i] when
// given, else position[rows[i]]); slots past n get node -1.
__device__ inline void part_load(const int32_t *__restrict__ rows, const int32_t *__restrict__ position,
                                 const int32_t *__restrict__ slot_node, int64_t i0, int64_t n,
                                 int32_t r[kPartItems], int32_t nid[kPartItems])
{
    if (i0 + kPartItems <= n) {
        const int4 rv = *(const int4 *)(rows + i0);
        r[0] = rv.x, r[1] = rv.y, r[2] = rv.z, r[3] = rv.w;
        if (slot_node) {
            const int4 nv = *(const int4 *)(slot_node + i0);
            nid[0] = nv.x, nid[1] = nv.y, nid[2] = nv.z, nid[3] = nv.w;
        }
    } else {
#pragma unroll
        for (int k = 0; k < kPartItems; ++k) {
            r[k] = i0 + k < n ? rows[i0 + k] : 0;
            if (slot_node) nid[k] = i0 + k < n ? slot_node[i0 + k] : -1;
        }
    }
    if (!slot_node) {
#pragma unroll
        for (int k = 0; k < kPartItems; ++k) nid[k] = i0 + k < n ? position[r[k]] : -1;
    }
}

// The root level's slots: slot i holds row i, all in node 0 (no arrays read).
__device__ inline void part_root(int64_t i0, int64_t n, int32_t r[kPartItems], int32_t nid[kPartItems])
{
#pragma unroll
    for (int k = 0; k < kPartItems; ++k) {
        r[k] = i0 + k < n ? (int32_t)(i0 + k) : 0;
        nid[k] = i0 + k < n ? 0 : -1;
    }
}

// The split choice of one node, made by one wave from the node's candidates
// (one per feature): the highest gain, equal gains to the lowest feature; the
// node splits when that gain is positive.  Returns {split, feature,
// split_bin, default_left} (all lanes).  write: record the choice in the
// node (lane 0).
__device__ inline int4 wave_decide(const EvalCand *__restrict__ cand, int32_t m, DevNode *__restrict__ nodes,
                                   int32_t id, bool write)
{
    const int lane = threadIdx.x & 63;
    const DevNode &nd = nodes[id];
    const EvalCand *c = cand + (int64_t)nd.slot * m;
    int32_t bi = -1;
    double bg = 0.0;
    for (int32_t f = lane; f < m; f += 64) {
        const EvalCand &o = c[f];
        if (o.valid && (bi < 0 || o.gain > bg)) {
            bi = f;
            bg = o.gain;
        }
    }
    const double mx = wave_max_f64(bi >= 0 ? bg : -__builtin_inf());
    const int32_t best = wave_min<int32_t>((bi >= 0 && bg == mx) ? bi : 0x7fffffff);
    if (best == 0x7fffffff) return make_int4(0, 0, 0, 0);
    const EvalCand b = c[best];
    if (!(b.gain > 0.0)) return make_int4(0, 0, 0, 0);
    if (write && lane == 0) {
        DevNode &d = nodes[id];
        d.split = 1;
        d.feature = b.feature;
        d.split_bin = b.split_bin;
        d.default_left = b.default_left;
        d.gain = b.gain;
        d.left_g = b.lg;
        d.left_h = b.lh;
        d.right_g = nd.sum_g - b.lg;
        d.right_h = nd.sum_h - b.lh;
    }
    return make_int4(1, b.feature, b.split_bin, b.default_left);
}

// Left flags of each slot and the count of each tile (the scan's first
// pass).  kChoose: the split records are not yet in the node table; each
// wave chooses the splits of the level's nodes among its slots from their
// candidates, and the wave holding a node's first slot records the choice
// (a node without slots cannot split).
template <bool kChoose, bool kCount>
__global__ void __launch_bounds__(kPartThreads)
    k_part_flags_tiles(const int32_t *__restrict__ rows, int64_t n, const uint32_t *__restrict__ page, Geo geo,
                       const int32_t *__restrict__ position, const int32_t *__restrict__ slot_node,
                       DevNode *__restrict__ nodes, uint8_t *__restrict__ flags,
                       int32_t *__restrict__ tile_cnt, LevelChoice lc, SlotTable stbl, ColCopy cols,
                       int32_t root)
{
    __shared__ int32_t red[kPartThreads / 64];
    const int64_t i0 = (int64_t)blockIdx.x * kPartTile + (int64_t)threadIdx.x * kPartItems;
    int32_t r[kPartItems], nid[kPartItems];
    if (root)
        part_root(i0, n, r, nid);
    else
        part_load(rows, position, slot_node, i0, n, r, nid);
    int4 rec[kPartItems];  // {split, feature, split_bin, default_left}
    if (kChoose) {
        const int lane = threadIdx.x & 63;
        const int64_t w_lo = i0 - (int64_t)lane * kPartItems;  // the wave's first slot
        uint32_t need = 0;
#pragma unroll
        for (int k = 0; k < kPartItems; ++k) {
            rec[k] = make_int4(0, 0, 0, 0);
            if (nid[k] >= lc.lo && nid[k] < lc.hi) need |= 1u << k;
        }
        for (;;) {
            // the wave's smallest node still to choose for (uniform)
            int32_t t = 0x7fffffff;
#pragma unroll
            for (int k = 0; k < kPartItems; ++k)
                if ((need >> k) & 1u) t = min(t, nid[k]);
            t = wave_min(t);
            if (t == 0x7fffffff) break;
            const int64_t b0 = nodes[t].begin;
            const int4 ch = wave_decide(lc.cand, lc.m, nodes, t, b0 >= w_lo && b0 < w_lo + 64 * kPartItems);
#pragma unroll
            for (int k = 0; k < kPartItems; ++k)
                if (((need >> k) & 1u) && nid[k] == t) {
                    rec[k] = ch;
                    need &= ~(1u << k);
                }
        }
    } else {
#pragma unroll
        for (int k = 0; k < kPartItems; ++k)
            rec[k] = nid[k] >= 0 ? *(const int4 *)&nodes[nid[k]].split : make_int4(0, 0, 0, 0);
    }
    uint32_t f4 = 0;
    int32_t cnt = 0;
#pragma unroll
    for (int k = 0; k < kPartItems; ++k) {
        uint32_t f = 0;
        if (rec[k].x) {
            const uint32_t *row = page + (int64_t)r[k] * geo.row_words;
            int32_t b;
            if (cols.p) {
                const int64_t e = (int64_t)rec[k].y * cols.stride + r[k];
                if (cols.bytes == 1) {
                    // 255: missing; 254: bin 254 or above, read from the row
                    // when the split bin is above 254
                    const uint32_t s = ((const uint8_t *)cols.p)[e];
                    b = s == 255u ? -1 : (s == 254u && rec[k].z > 254 ? row_feature_bin(row, geo, rec[k].y) : (int32_t)s);
                } else {
                    const uint32_t s = ((const uint16_t *)cols.p)[e];
                    b = s == geo.null_sym ? -1 : (int32_t)s;
                }
            } else {
                if (stbl.col) {
                    const uint32_t se = stbl.col[(int64_t)stbl.feat_grp[rec[k].y] * stbl.rows + r[k]];
                    b = row_feature_bin_range(row, geo, rec[k].y, (int32_t)(se & 0xffu), (int32_t)(se >> 8));
                } else {
                    b = row_feature_bin(row, geo, rec[k].y);
                }
            }
            f = (b < 0) ? (rec[k].w != 0 ? 1u : 0u) : (b < rec[k].z ? 1u : 0u);
        }
        f4 |= f << (8 * k);
        cnt += (int32_t)f;
    }
    if (i0 + kPartItems <= n) {
        *(uint32_t *)(flags + i0) = f4;
    } else {
#pragma unroll
        for (int k = 0; k < kPartItems; ++k)
            if (i0 + k < n) flags[i0 + k] = (uint8_t)((f4 >> (8 * k)) & 1u);
    }
    if (kCount) {
        // the left flags of this tile before each node's first slot and up
        // to its last slot, written by the tile holding that slot (the plan
        // adds the counts of the tiles before); a node's slots are one run
        // of equal slot nodes
        const int32_t prev = i0 > 0 && i0 <= n ? (root ? 0 : slot_node[i0 - 1]) : -2;
        const int32_t next = i0 + kPartItems < n ? (root ? 0 : slot_node[i0 + kPartItems]) : -2;
        int32_t tot;
        int32_t pre = part_block_scan(cnt, red, &tot);
#pragma unroll
        for (int k = 0; k < kPartItems; ++k) {
            const int32_t f = (int32_t)((f4 >> (8 * k)) & 1u);
            if (i0 + k < n && nid[k] >= 0) {
                const int32_t lo = k == 0 ? prev : nid[k - 1];
                const int32_t hi = k == kPartItems - 1 ? next : nid[k + 1];
                if (lo != nid[k]) {
                    nodes[nid[k]].tile_b = (int32_t)blockIdx.x;
                    nodes[nid[k]].left_b = pre;
                }
                if (hi != nid[k]) {
                    nodes[nid[k]].tile_e = (int32_t)blockIdx.x;
                    nodes[nid[k]].left_e = pre + f;
                }
            }
            pre += f;
        }
        if (threadIdx.x == 0) tile_cnt[blockIdx.x] = tot;
        return;
    }
    cnt = wave_total(cnt);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = cnt;
    __syncthreads();
    if (threadIdx.x == 0) {
        int32_t t = 0;
        for (int w = 0; w < kPartThreads / 64; ++w) t += red[w];
        tile_cnt[blockIdx.x] = t;
    }
}

// Left flags before slot x: the counts of the tiles before x's tile plus the
// flags of that tile before x, summed by the 256 threads of the block.
constexpr int kBoundThreads = 256;

__device__ inline uint32_t byte_sum4(uint32_t v)
{
    return ((v & 0x01010101u) * 0x01010101u) >> 24;  // four 0/1 bytes
}

__device__ inline int64_t part_prefix(const uint8_t *__restrict__ flags, const int32_t *__restrict__ tile_cnt,
                                      int64_t x, long long *lds4)
{
    static_assert(kBoundThreads * 16 >= kPartTile, "one block covers a tile's flags, 16 per thread");
    const int64_t t = x / kPartTile, s = t * kPartTile;
    const int64_t j = s + (int64_t)threadIdx.x * 16;
    long long c = 0;
    if (j + 16 <= x) {
        const uint4 v = *(const uint4 *)(flags + j);
        c = byte_sum4(v.x) + byte_sum4(v.y) + byte_sum4(v.z) + byte_sum4(v.w);
    } else {
        for (int64_t k = j; k < x; ++k) c += flags[k];
    }
    for (int64_t k = threadIdx.x; k < t; k += kBoundThreads) c += tile_cnt[k];
    c = wave_total(c);
    __syncthreads();
    if ((threadIdx.x & 63) == 0) lds4[threadIdx.x >> 6] = c;
    __syncthreads();
    return lds4[0] + lds4[1] + lds4[2] + lds4[3];
}

// For every splitting node of the list: the left flags before its segment
// and the count of its rows that go left.  One block per node.
__global__ void __launch_bounds__(kBoundThreads)
    k_part_bounds(const EvalNode *__restrict__ list, const int32_t *__restrict__ n_list_d, int32_t n_list,
                  DevNode *__restrict__ nodes, const uint8_t *__restrict__ flags,
                  const int32_t *__restrict__ tile_cnt)
{
    __shared__ long long lds4[kBoundThreads / 64];
    const int32_t count = n_list_d ? *n_list_d : n_list;
    if ((int32_t)blockIdx.x >= count) return;
    const int32_t nid = list ? list[blockIdx.x].heap : (int32_t)blockIdx.x;
    DevNode &d = nodes[nid];
    if (!d.split) return;
    const int64_t pb = part_prefix(flags, tile_cnt, d.begin, lds4);
    const int64_t pe = part_prefix(flags, tile_cnt, d.end, lds4);
    if (threadIdx.x == 0) {
        d.pleft = pb;
        d.nleft = pe - pb;
    }
}

// Stable scatter: the slot's exclusive left count comes from the tile offset
// and a block scan; a splitting node's left rows go to the front of its
// segment, the others after them, both in slot order.
__global__ void __launch_bounds__(kPartThreads)
    k_part_scatter(const int32_t *__restrict__ rows, int64_t n, const uint8_t *__restrict__ flags,
                   const int32_t *__restrict__ tile_cnt, const int32_t *__restrict__ position,
                   int32_t *__restrict__ position_out,
                   const int32_t *__restrict__ slot_node, int32_t *__restrict__ slot_node_out,
                   const DevNode *__restrict__ nodes, int32_t *__restrict__ rows_out)
{
    __shared__ int32_t lds16[kPartThreads / 64];
    const int64_t i0 = (int64_t)blockIdx.x * kPartTile + (int64_t)threadIdx.x * kPartItems;
    int32_t r[kPartItems], nid[kPartItems];
    part_load(rows, position, slot_node, i0, n, r, nid);
    uint32_t f4 = 0;
    if (i0 + kPartItems <= n) {
        f4 = *(const uint32_t *)(flags + i0);
    } else {
#pragma unroll
        for (int k = 0; k < kPartItems; ++k)
            if (i0 + k < n) f4 |= (uint32_t)flags[i0 + k] << (8 * k);
    }
    const int32_t mine = (int32_t)((f4 & 1u) + ((f4 >> 8) & 1u) + ((f4 >> 16) & 1u) + ((f4 >> 24) & 1u));
    // left flags of the tiles before this one (their counts, summed here)
    __shared__ long long tl16[kPartThreads / 64];
    long long before = 0;
    for (int64_t k = threadIdx.x; k < (int64_t)blockIdx.x; k += kPartThreads) before += tile_cnt[k];
    before = wave_total(before);
    if ((threadIdx.x & 63) == 0) tl16[threadIdx.x >> 6] = before;
    int32_t total;
    const int32_t in_tile = part_block_scan(mine, lds16, &total);  // synchronizes the block
    before = 0;
#pragma unroll
    for (int w = 0; w < kPartThreads / 64; ++w) before += tl16[w];
    int64_t P = before + in_tile;
#pragma unroll
    for (int k = 0; k < kPartItems; ++k) {
        const int64_t i = i0 + k;
        const uint32_t f = (f4 >> (8 * k)) & 1u;
        if (i < n) {
            int64_t dest = i;
            int32_t child = nid[k];
            if (nid[k] >= 0) {
                const DevNode &nd = nodes[nid[k]];
                const int4 rec = *(const int4 *)&nd.split;
                if (rec.x) {
                    const int64_t pl = P - nd.pleft;
                    if (f) {
                        dest = nd.begin + pl;
                        child = nd.left_child;
                    } else {
                        dest = nd.begin + nd.nleft + (i - nd.begin - pl);
                        child = nd.right_child;
                    }
                    if (position_out) position_out[r[k]] = child;
                }
            }
            rows_out[dest] = r[k];
            if (slot_node_out) slot_node_out[dest] = child;
        }
        P += f;
    }
}

// The tree driver's scatter, which also takes the place of k_part_bounds: a
// splitting node's left rows go to the front of its segment in slot order
// and its right rows to the back in reverse slot order, so no block needs a
// node's total left count.  The left flags before a node's first slot come
// from this tile's scan when the node starts in the tile; the one node that
// starts in an earlier tile (the node of the tile's first slot) gets them
// from the tile counts before its first tile and that tile's flags.  The
// order of rows within a node enters no result.  Block 0 is the level's plan (plan_impl.h), which
// reads only the node records and the boundary counts of the flags pass and
// writes the nodes' left counts and the children's records, which no other
// block reads; the tiles are blocks 1.. .
__global__ void __launch_bounds__(kPartThreads)
    k_part_scatter_rev(const int32_t *__restrict__ rows, int64_t n, const uint8_t *__restrict__ flags,
                       const int32_t *__restrict__ tile_cnt, const long long *__restrict__ tile_off,
                       const int32_t *__restrict__ slot_node, int32_t *__restrict__ slot_node_out,
                       DevNode *__restrict__ nodes, int32_t *__restrict__ rows_out, int32_t root, PlanArgs pa)
{
    if (blockIdx.x == 0) {
        pa.tile_cnt = tile_cnt;
        pa.tile_off = tile_off;
        pa.tiles = (n + kPartTile - 1) / kPartTile;
        plan_level_block<kPartThreads>(nodes, pa);
        return;
    }
    const int64_t tile = (int64_t)blockIdx.x - 1;
    __shared__ int32_t lds16[kPartThreads / 64];
    __shared__ long long s_red[2][kPartThreads / 64];
    __shared__ int32_t s_pref[kPartThreads];  // left flags of the tile before each thread's slots
    __shared__ uint32_t s_f4[kPartThreads];   // each thread's four flags, one per byte
    const int64_t ts = tile * kPartTile;
    const int64_t i0 = ts + (int64_t)threadIdx.x * kPartItems;
    int32_t r[kPartItems], nid[kPartItems];
    if (root)
        part_root(i0, n, r, nid);
    else
        part_load(rows, nullptr, slot_node, i0, n, r, nid);
    uint32_t f4 = 0;
    if (i0 + kPartItems <= n) {
        f4 = *(const uint32_t *)(flags + i0);
    } else {
#pragma unroll
        for (int k = 0; k < kPartItems; ++k)
            if (i0 + k < n) f4 |= (uint32_t)flags[i0 + k] << (8 * k);
    }
    const int32_t mine = (int32_t)((f4 & 1u) + ((f4 >> 8) & 1u) + ((f4 >> 16) & 1u) + ((f4 >> 24) & 1u));
    // the node of the tile's first slot, when it starts in an earlier tile
    const int32_t n0 = root ? 0 : slot_node[ts];
    const int64_t b0 = n0 >= 0 ? nodes[n0].begin : ts;
    const bool ext = b0 < ts;
    const int64_t tb = b0 / kPartTile;  // its first tile
    // left flags before this tile and before b0: tile counts, plus the
    // flags of tile tb before b0
    long long before = 0, before_b = 0;
    if (tile_off) {
        // exclusive tile offsets: the first wave's first lane takes both
        if (threadIdx.x == 0) {
            before = tile_off[tile];
            before_b = tile_off[tb];
        }
    } else {
        for (int64_t k = threadIdx.x; k < tile; k += kPartThreads) {
            const int32_t v = tile_cnt[k];
            before += v;
            before_b += k < tb ? v : 0;
        }
    }
    if (ext) {
        const int64_t j = tb * kPartTile + (int64_t)threadIdx.x * kPartItems;
#pragma unroll
        for (int k = 0; k < kPartItems; ++k) before_b += j + k < b0 ? flags[j + k] : 0;
    }
    before = wave_total(before);
    before_b = wave_total(before_b);
    if ((threadIdx.x & 63) == 0) {
        s_red[0][threadIdx.x >> 6] = before;
        s_red[1][threadIdx.x >> 6] = before_b;
    }
    int32_t total;
    const int32_t in_tile = part_block_scan(mine, lds16, &total);  // synchronizes the block
    s_pref[threadIdx.x] = in_tile;
    s_f4[threadIdx.x] = f4;
    before = 0;
    before_b = 0;
#pragma unroll
    for (int w = 0; w < kPartThreads / 64; ++w) {
        before += s_red[0][w];
        before_b += s_red[1][w];
    }
    __syncthreads();
    long long P = before + in_tile;  // left flags before slot i (all slots)
#pragma unroll
    for (int k = 0; k < kPartItems; ++k) {
        const int64_t i = i0 + k;
        const uint32_t f = (f4 >> (8 * k)) & 1u;
        if (i < n) {
            int64_t dest = i;
            int32_t child = nid[k];
            if (nid[k] >= 0) {
                DevNode &nd = nodes[nid[k]];
                const int4 rec = *(const int4 *)&nd.split;
                if (rec.x) {
                    const int64_t begin = nd.begin, end = nd.end;
                    long long pl;  // left flags before the node's first slot
                    if (begin < ts) {
                        pl = before_b;
                    } else {
                        const int o = (int)(begin - ts), th = o / kPartItems, kk = o % kPartItems;
                        const uint32_t fb = s_f4[th] & ((1u << (8 * kk)) - 1u);
                        pl = before + s_pref[th] + (long long)((fb & 1u) + ((fb >> 8) & 1u) + ((fb >> 16) & 1u));
                    }
                    const long long lb = P - pl;  // the node's left rows before slot i
                    if (f) {
                        dest = begin + lb;
                        child = nd.left_child;
                    } else {
                        dest = end - 1 - ((i - begin) - lb);
                        child = nd.right_child;
                    }
                }
            }
            rows_out[dest] = r[k];
            slot_node_out[dest] = child;
        }
        P += f;
    }
}

// Exclusive offsets of the partition's tile counts, by one block: each
// thread sums a contiguous run of counts, the block scans the run totals,
// and each thread writes its run's offsets.
constexpr int kTileScanThreads = 1024;
constexpr int64_t kScanTilesAbove = 2048;
static_assert(kScanTilesAbove <= kPlanScanTiles, "the plan block scans the tile counts that have no offsets");

__global__ void __launch_bounds__(kTileScanThreads)
    k_tile_offsets(const int32_t *__restrict__ cnt, int64_t tiles, long long *__restrict__ off)
{
    __shared__ long long s_w[kTileScanThreads / 64];
    const int64_t per = (tiles + kTileScanThreads - 1) / kTileScanThreads;
    const int64_t a = min<int64_t>(tiles, (int64_t)threadIdx.x * per), b = min<int64_t>(tiles, a + per);
    constexpr int kHeld = 16;  // runs this short are loaded at once (all loads in flight)
    int32_t v[kHeld];
    long long run = 0;
    if (per <= kHeld) {
#pragma unroll
        for (int j = 0; j < kHeld; ++j) v[j] = a + j < b ? cnt[a + j] : 0;
#pragma unroll
        for (int j = 0; j < kHeld; ++j) run += v[j];
    } else {
        for (int64_t k = a; k < b; ++k) run += cnt[k];
    }
    // inclusive scan of the run totals: within the wave, then over waves
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    const long long x = wave_incl_sum(run);
    if (lane == 63) s_w[wid] = x;
    __syncthreads();
    long long base = x - run;
    for (int w = 0; w < wid; ++w) base += s_w[w];
    if (per <= kHeld) {
#pragma unroll
        for (int j = 0; j < kHeld; ++j)
            if (a + j < b) {
                off[a + j] = base;
                base += v[j];
            }
    } else {
        for (int64_t k = a; k < b; ++k) {
            off[k] = base;
            base += cnt[k];
        }
    }
}

// Column copy of a dense page (ColCopy: entry (f, r) at f * stride + r).  A
// block stages 256 consecutive rows in LDS (an odd pitch keeps the threads'
// reads on distinct banks) and writes each feature's 256 entries with
// consecutive stores.
constexpr int kColRows = 256;

template <typename T>
__global__ void __launch_bounds__(kColRows)
    k_page_columns(const uint32_t *__restrict__ page, int64_t n, int32_t row_words, int32_t m, int32_t w,
                   uint32_t mask, uint32_t null_sym, T *__restrict__ cols, int64_t stride)
{
    extern __shared__ uint32_t rows_l[];  // kColRows x (row_words | 1)
    const int64_t r0 = (int64_t)blockIdx.x * kColRows;
    const int32_t nr = (int32_t)min<int64_t>(kColRows, n - r0);
    const int32_t nw = nr * row_words, lw = row_words | 1;
    const uint32_t *src = page + r0 * row_words;
    for (int32_t k0 = 0; k0 < nw; k0 += kColRows * 8) {
        uint32_t v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int32_t k = k0 + j * kColRows + (int32_t)threadIdx.x;
            v[j] = k < nw ? src[k] : 0u;
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int32_t k = k0 + j * kColRows + (int32_t)threadIdx.x;
            if (k < nw) {
                const int32_t rr = k / row_words;
                rows_l[rr * lw + (k - rr * row_words)] = v[j];
            }
        }
    }
    __syncthreads();
    if ((int32_t)threadIdx.x >= nr) return;
    const uint32_t *row = rows_l + threadIdx.x * lw;
    T *dst = cols + r0 + threadIdx.x;
    for (int32_t f = 0; f < m; ++f) {
        const uint32_t bit = (uint32_t)f * (uint32_t)w, k = bit >> 5;
        const uint32_t hi = k + 1 < (uint32_t)row_words ? row[k + 1] : 0u;
        const uint32_t sym = __builtin_amdgcn_alignbit(hi, row[k], bit & 31u) & mask;
        if constexpr (sizeof(T) == 1)
            dst[(int64_t)f * stride] = col_byte(sym, null_sym);
        else
            dst[(int64_t)f * stride] = (T)sym;
    }
}

bool split_columns_fit(const gbt_matrix *mx) { return !mx->sparse && mx->w <= 16 && mx->row_words <= 64; }

int32_t split_columns_bytes(const gbt_matrix *mx)
{
    int32_t max_bins = 0;
    for (int32_t f = 0; f < mx->m; ++f) max_bins = std::max(max_bins, mx->bin_ptr_h[f + 1] - mx->bin_ptr_h[f]);
    return max_bins <= 256 ? 1 : 2;
}

gbt_status split_columns(gbt_ctx *c, const gbt_matrix *mx, const uint32_t *page, int64_t n, const ColCopy &cols)
{
    GBT_CHECK(split_columns_fit(mx), "column copy of a page with %d-bit symbols", mx->w);
    GBT_CHECK((cols.bytes == 1 || cols.bytes == 2) && cols.stride >= n, "column copy layout");
    if (n <= 0) return GBT_OK;
    const uint32_t mask = mx->w >= 32 ? 0xffffffffu : ((1u << mx->w) - 1u);
    const uint32_t null_sym = mx->has_missing ? mx->null_sym : 0xffffffffu;
    const size_t lds = (size_t)kColRows * (mx->row_words | 1) * 4;
    const unsigned grid = (unsigned)((n + kColRows - 1) / kColRows);
    if (cols.bytes == 1)
        k_page_columns<uint8_t><<<grid, kColRows, lds, c->stream>>>(page, n, mx->row_words, mx->m, mx->w, mask,
                                                                   null_sym, (uint8_t *)cols.p, cols.stride);
    else
        k_page_columns<uint16_t><<<grid, kColRows, lds, c->stream>>>(page, n, mx->row_words, mx->m, mx->w, mask,
                                                                    null_sym, (uint16_t *)cols.p, cols.stride);
    GBT_LAUNCHED();
    return GBT_OK;
}

gbt_status partition_rev_impl(gbt_ctx *c, const gbt_matrix *mx, const uint32_t *page, const int32_t *rows,
                              int64_t n, const int32_t *slot_node, int32_t *slot_node_out, DevNode *nodes,
                              int32_t *rows_out, const LevelChoice *choice, const SlotTable *stbl,
                              const ColCopy &cols, const PlanArgs &plan, bool order, bool root)
{
    if (n == 0) return GBT_OK;
    const SlotTable st = stbl ? *stbl : SlotTable{nullptr, nullptr, nullptr, 0, 0, 0};
    GBT_CHECK(n < ((int64_t)1 << 31) - 1, "partition of %lld rows (limit 2^31-2)", (long long)n);
    uint8_t *flags;
    GBT_TRY(scratch_t(c, kScrPartFlags, (size_t)n + 16, &flags));
    const int64_t tiles = (n + kPartTile - 1) / kPartTile;
    int32_t *tile_cnt;
    GBT_TRY(scratch_t(c, kScrScan, (size_t)tiles + 1, &tile_cnt));
    if (choice)
        k_part_flags_tiles<true, true><<<(unsigned)tiles, kPartThreads, 0, c->stream>>>(
            rows, n, page, geo_of(mx), nullptr, slot_node, nodes, flags, tile_cnt, *choice, st, cols, root ? 1 : 0);
    else
        k_part_flags_tiles<false, true><<<(unsigned)tiles, kPartThreads, 0, c->stream>>>(
            rows, n, page, geo_of(mx), nullptr, slot_node, nodes, flags, tile_cnt, LevelChoice{}, st, cols,
            root ? 1 : 0);
    GBT_LAUNCHED();
    // many tiles: one block scans the tile counts first, instead of every
    // block summing the counts before it
    long long *tile_off = nullptr;
    if (tiles > kScanTilesAbove) {
        GBT_TRY(scratch_t(c, kScrPartPos, (size_t)tiles, &tile_off));
        k_tile_offsets<<<1, kTileScanThreads, 0, c->stream>>>(tile_cnt, tiles, tile_off);
        GBT_LAUNCHED();
    }
    // without the row order only the plan block runs
    k_part_scatter_rev<<<(unsigned)((order ? tiles : 0) + 1), kPartThreads, 0, c->stream>>>(
        rows, n, flags, tile_cnt, tile_off, slot_node, slot_node_out, nodes, rows_out, root ? 1 : 0, plan);
    GBT_LAUNCHED();
    return GBT_OK;
}

gbt_status partition_impl(gbt_ctx *c, const gbt_matrix *mx, const uint32_t *page, const int32_t *rows,
                          int64_t n, int32_t *position, const int32_t *slot_node, int32_t *slot_node_out,
                          DevNode *nodes, const EvalNode *list, const int32_t *n_list_d, int32_t n_list,
                          int32_t *rows_out)
{
    if (n == 0) return GBT_OK;
    GBT_CHECK(n < ((int64_t)1 << 31) - 1, "partition of %lld rows (limit 2^31-2)", (long long)n);
    uint8_t *flags;
    GBT_TRY(scratch_t(c, kScrPartFlags, (size_t)n + 16, &flags));
    Geo geo = geo_of(mx);
    const int64_t tiles = (n + kPartTile - 1) / kPartTile;
    int32_t *tile_off;
    GBT_TRY(scratch_t(c, kScrScan, (size_t)tiles + 1, &tile_off));
    // tile_off receives each tile's left count; the bounds and the scatter
    // sum the counts before their tiles themselves
    k_part_flags_tiles<false, false><<<(unsigned)tiles, kPartThreads, 0, c->stream>>>(rows, n, page, geo, position, slot_node,
                                                                       nodes, flags, tile_off, LevelChoice{},
                                                                       SlotTable{nullptr, nullptr, nullptr, 0, 0, 0},
                                                                       ColCopy{}, 0);
    GBT_LAUNCHED();
    if (n_list > 0) {
        k_part_bounds<<<(unsigned)n_list, kBoundThreads, 0, c->stream>>>(list, n_list_d, n_list, nodes, flags,
                                                                         tile_off);
        GBT_LAUNCHED();
    }
    // with slot nodes kept the caller derives positions at the end; without
    // them, positions are the partition's output
    k_part_scatter<<<(unsigned)tiles, kPartThreads, 0, c->stream>>>(
        rows, n, flags, tile_off, position, slot_node_out ? nullptr : position, slot_node, slot_node_out, nodes,
        rows_out);
    GBT_LAUNCHED();
    return GBT_OK;
}

// ------------------------------------------------------------ public calls
// Work tables of gbt_eval_splits and gbt_partition built on the device from
// the caller's device arrays.

constexpr unsigned kSegBlocks = 64;  // blocks per node segment in k_slot_of_segments

__global__ void k_zero_i32(int32_t *__restrict__ p, int32_t n)
{
    if ((int32_t)threadIdx.x < n) p[threadIdx.x] = 0;
}

__global__ void k_copy_i32(const int32_t *__restrict__ src, int32_t *__restrict__ dst, int32_t n)
{
    if ((int32_t)threadIdx.x < n) dst[threadIdx.x] = src[threadIdx.x];
}

__global__ void k_fill_i32(int32_t *__restrict__ p, int64_t n, int32_t v)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = v;
}

__global__ void k_eval_nodes(const int64_t *__restrict__ sums, const int32_t *__restrict__ slots, int32_t n,
                             EvalNode *__restrict__ out)
{
    const int32_t k = (int32_t)(blockIdx.x * blockDim.x + threadIdx.x);
    if (k >= n) return;
    EvalNode e;
    e.sum_g = sums[2 * (int64_t)k];
    e.sum_h = sums[2 * (int64_t)k + 1];
    e.slot = slots[k];
    e.heap = k;
    out[k] = e;
}

// Node k of the partition from split[k], seg[k] and child[2k], child[2k+1].
// A segment outside [0, n_rows] is clamped into it and a split feature
// outside [0, m) does not split: either adds one to *bad.
__global__ void k_part_nodes(const gbt_split *__restrict__ split, const gbt_seg *__restrict__ seg,
                             const int32_t *__restrict__ child, int32_t n_nodes, int64_t n_rows, int32_t m,
                             DevNode *__restrict__ nodes, int32_t *__restrict__ bad)
{
    const int32_t k = (int32_t)(blockIdx.x * blockDim.x + threadIdx.x);
    if (k >= n_nodes) return;
    const gbt_seg sg = seg[k];
    const gbt_split sp = split[k];
    bool ok = true;
    int64_t b = sg.begin, e = sg.end;
    if (b < 0 || b > e || e > n_rows) {
        ok = false;
        b = b < 0 ? 0 : (b > n_rows ? n_rows : b);
        e = e < b ? b : (e > n_rows ? n_rows : e);
    }
    bool splits = sp.valid != 0;
    if (splits && (sp.feature < 0 || sp.feature >= m)) {
        ok = false;
        splits = false;
    }
    DevNode d = {};
    d.begin = b;
    d.end = e;
    d.present = 1;
    d.split = splits ? 1 : 0;
    d.feature = splits ? sp.feature : 0;
    d.split_bin = splits ? sp.split_bin : 0;
    d.default_left = splits ? sp.default_left : 0;
    d.left_child = child[2 * (int64_t)k];
    d.right_child = child[2 * (int64_t)k + 1];
    nodes[k] = d;
    if (!ok) atomicAdd(bad, 1);
}

// slot_node[i] = k for every slot i of node k's segment (blockIdx.x = k,
// gridDim.y blocks stride over it); a slot that two segments claim adds one
// to *bad.
__global__ void k_slot_of_segments(const DevNode *__restrict__ nodes, int32_t *__restrict__ slot_node,
                                   int32_t *__restrict__ bad)
{
    const int32_t k = (int32_t)blockIdx.x;
    const int64_t b = nodes[k].begin, e = nodes[k].end;
    const int64_t step = (int64_t)gridDim.y * blockDim.x;
    for (int64_t i = b + (int64_t)blockIdx.y * blockDim.x + threadIdx.x; i < e; i += step)
        if (atomicExch(&slot_node[i], k) != -1) atomicAdd(bad, 1);
}

// The child segments of node k: [begin, begin + nleft) and [begin + nleft,
// end) of a splitting node; the whole segment left of one that does not split.
__global__ void k_child_segments(const DevNode *__restrict__ nodes, int32_t n_nodes, int64_t n_rows,
                                 gbt_seg *__restrict__ out)
{
    const int32_t k = (int32_t)(blockIdx.x * blockDim.x + threadIdx.x);
    if (k >= n_nodes) return;
    const DevNode &d = nodes[k];
    const int64_t nl = (d.split && n_rows) ? d.nleft : d.end - d.begin;
    gbt_seg l, r;
    l.node_slot = d.left_child;
    l.pad0 = 0;
    l.begin = d.begin;
    l.end = d.begin + nl;
    r.node_slot = d.right_child;
    r.pad0 = 0;
    r.begin = d.begin + nl;
    r.end = d.end;
    out[2 * (int64_t)k] = l;
    out[2 * (int64_t)k + 1] = r;
}

}  // namespace gbt

using namespace gbt;

extern "C" {

gbt_status gbt_eval_splits(gbt_ctx *c, const gbt_matrix *layout, const int64_t *hist_d,
                           const int64_t *node_sum_d, const int32_t *node_slot_d, int32_t n_nodes,
                           const gbt_train_params *tp, int32_t exp_g, int32_t exp_h, gbt_split *out_d)
{
    GBT_CHECK(c && layout && tp && out_d, "gbt_eval_splits: NULL argument");
    GBT_CHECK(n_nodes >= 0, "negative node count");
    if (n_nodes == 0) return GBT_OK;
    GBT_CHECK(hist_d && node_sum_d && node_slot_d, "gbt_eval_splits: NULL input");
    GBT_TRY(set_device(c));
    EvalNode *nodes_d;
    GBT_TRY(scratch_t(c, kScrEvalNodes, (size_t)n_nodes, &nodes_d));
    k_eval_nodes<<<(unsigned)((n_nodes + 255) / 256), 256, 0, c->stream>>>(node_sum_d, node_slot_d, n_nodes,
                                                                          nodes_d);
    GBT_LAUNCHED();
    EvalParams ep{tp->lambda, tp->gamma, tp->min_child_weight, exp_g, exp_h, nullptr};
    return eval_impl(c, layout, hist_d, nodes_d, n_nodes, ep, out_d);
}

gbt_status gbt_partition(gbt_ctx *c, const gbt_matrix *layout, const uint32_t *page_d,
                         const gbt_split *split_d, const gbt_seg *seg_d, const int32_t *child_d,
                         int32_t n_nodes, int32_t *rows_d, int32_t *rows_tmp_d, int64_t n_rows,
                         int32_t *position_d, gbt_seg *seg_out_d, int32_t *status_d)
{
    GBT_CHECK(c && layout && page_d && rows_d && rows_tmp_d && position_d, "gbt_partition: NULL argument");
    GBT_CHECK(n_nodes >= 0 && n_rows >= 0, "negative sizes");
    GBT_CHECK(n_nodes == 0 || (split_d && seg_d && child_d && seg_out_d), "gbt_partition: NULL node arrays");
    GBT_CHECK(n_rows < ((int64_t)1 << 31) - 1, "partition of %lld rows (limit 2^31-2)", (long long)n_rows);
    GBT_CHECK(((uintptr_t)rows_d & 15) == 0 && ((uintptr_t)rows_tmp_d & 15) == 0,
              "gbt_partition: rows_d and rows_tmp_d must be 16-byte aligned");
    GBT_TRY(set_device(c));
    DevNode *nodes_d;
    int32_t *slot_node, *bad;
    GBT_TRY(scratch_t(c, kScrNodes, (size_t)std::max(n_nodes, 1), &nodes_d));
    GBT_TRY(scratch_t(c, kScrSlotNode, (size_t)std::max<int64_t>(n_rows, 1), &slot_node));
    GBT_TRY(scratch_t(c, kScrEvalNodes, 4, &bad));
    k_zero_i32<<<1, 64, 0, c->stream>>>(bad, 1);
    GBT_LAUNCHED();
    if (n_nodes) {
        k_part_nodes<<<(unsigned)((n_nodes + 255) / 256), 256, 0, c->stream>>>(split_d, seg_d, child_d, n_nodes,
                                                                               n_rows, layout->m, nodes_d, bad);
        GBT_LAUNCHED();
    }
    if (n_rows) {
        k_fill_i32<<<(unsigned)((n_rows + 255) / 256), 256, 0, c->stream>>>(slot_node, n_rows, -1);
        GBT_LAUNCHED();
        if (n_nodes) {
            // each node's (clamped) segment, strided over by up to kSegBlocks blocks
            const unsigned per = (unsigned)std::max<int64_t>(1, std::min<int64_t>(kSegBlocks, 65536 / n_nodes));
            k_slot_of_segments<<<dim3((unsigned)n_nodes, per), 256, 0, c->stream>>>(nodes_d, slot_node, bad);
            GBT_LAUNCHED();
        }
    }
    GBT_TRY(partition_impl(c, layout, page_d, rows_d, n_rows, position_d, slot_node, nullptr, nodes_d, nullptr,
                           nullptr, n_nodes, rows_tmp_d));
    if (n_rows)
        GBT_HIP(hipMemcpyAsync(rows_d, rows_tmp_d, (size_t)n_rows * 4, hipMemcpyDeviceToDevice, c->stream));
    if (n_nodes) {
        k_child_segments<<<(unsigned)((n_nodes + 255) / 256), 256, 0, c->stream>>>(nodes_d, n_nodes, n_rows,
                                                                                   seg_out_d);
        GBT_LAUNCHED();
    }
    if (status_d) {
        k_copy_i32<<<1, 64, 0, c->stream>>>(bad, status_d, 1);
        GBT_LAUNCHED();
    }
    return GBT_OK;
}

}  // extern "C"
