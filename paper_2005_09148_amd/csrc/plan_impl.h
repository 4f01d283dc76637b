// plan_impl.h -- the level plan of the tree driver (Alg. 1's level loop),
// run by one block of T threads after a level's partition: the child
// segments and sums of every split node from the partition's left count
// (nleft), then, when `plan` is set, the plan of the next level: the list of
// present children in heap order with their histogram slots, and for each
// split parent the smaller child to build (chunked into work items) with the
// larger one as parent minus it.  The chunk size is chosen so that the level
// has at most `items` work items per feature group (one per workgroup slot)
// while it builds at most items / 2 nodes, and at most items plus its node
// count beyond that.
#pragma once

#include "split_impl.h"
#include "wave_impl.h"

namespace gbt {

constexpr int64_t kMinChunk = 1024;
// tile counts the plan block scans itself (more come with their offsets)
constexpr int32_t kPlanScanTiles = 2048;

// What the plan needs of one split parent, all from the parent's record.
struct PlanNode {
    int64_t begin, nl, nr;  // segment start, left and right row counts
    long long lg, lh, rg, rh;
    int32_t p, slot, split, pad0;
};

__device__ inline PlanNode plan_node(const EvalNode *__restrict__ cur, const DevNode *__restrict__ nodes, int32_t t)
{
    PlanNode x;
    x.p = cur[t].heap;
    x.slot = cur[t].slot;
    const DevNode &d = nodes[x.p];
    x.split = d.split;
    x.begin = d.begin;
    x.nl = d.nleft;
    x.nr = d.end - d.begin - d.nleft;
    x.lg = d.left_g;
    x.lh = d.left_h;
    x.rg = d.right_g;
    x.rh = d.right_h;
    x.pad0 = 0;
    return x;
}

// Exclusive scan across a block of T threads; *total receives the sum.
template <int T>
__device__ inline int32_t plan_block_scan(int32_t v, int32_t *lds, int32_t *total)
{
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    const int32_t x = wave_incl_sum(v);
    __syncthreads();
    if (lane == 63) lds[wid] = x;
    __syncthreads();
    int32_t off = 0, tot = 0;
    for (int w = 0; w < T / 64; ++w) {
        if (w < wid) off += lds[w];
        tot += lds[w];
    }
    *total = tot;
    return x - v + off;
}

// Eq. 6 scaled by the learning rate, for every present node that does not
// split: leaf = (float)((-G/(H+lambda)) * eta).
__device__ inline float leaf_of(long long Qg, long long Qh, int32_t eg, int32_t eh, double lambda, double eta)
{
    double G = ldexp((double)Qg, -eg), H = ldexp((double)Qh, -eh);
    double w = -G / (H + lambda);
    return (float)(w * eta);
}

// Node i's leaf value, and its entry in the compact form of the tree used by
// the row walk: {feature, split_bin << 2 | default_left << 1 | splits}.
__device__ inline void leaf_entry(const DevNode *__restrict__ nodes, int32_t i, int32_t eg, int32_t eh,
                                  double lambda, double eta, float *__restrict__ leaf, uint2 *__restrict__ compact)
{
    const DevNode d = nodes[i];
    leaf[i] = (d.present && !d.split) ? leaf_of(d.sum_g, d.sum_h, eg, eh, lambda, eta) : 0.0f;
    compact[i] = d.split ? make_uint2((uint32_t)d.feature, ((uint32_t)d.split_bin << 2) |
                                                               ((d.default_left ? 1u : 0u) << 1) | 1u)
                         : make_uint2(0u, 0u);
}

// The tree's leaves, made by the last level's plan (leaf == NULL: none).
struct LeafArgs {
    float *leaf;
    uint2 *compact;
    const int32_t *e_dev;  // {e_g, e_h}
    double lambda, eta;
    int32_t n_nodes;
    int32_t pad0;
};

struct PlanArgs {
    const EvalNode *cur;     // the level's nodes (count *n_cur_d)
    const int32_t *n_cur_d;
    int32_t plan;            // plan the next level's histograms
    int32_t items;           // work items per feature group to aim for
    EvalNode *next;          // out: the next level's nodes
    int32_t *n_next_d;
    HistWork *work;          // out: its histogram work items
    int32_t *n_work_d;
    HistReduce *red;         // out: its reduce items (one per built node)
    int32_t *n_red_d;
    unsigned long long *stat;  // rows built, histograms built
    // the partition's left flags per tile (and their exclusive offsets, or
    // NULL when there are at most kPlanScanTiles tiles): each node's left
    // count from its boundary prefixes (DevNode::tile_b ...); when tile_cnt
    // is NULL, DevNode::nleft already holds it
    const int32_t *tile_cnt;
    const long long *tile_off;
    int64_t tiles;
    LeafArgs lv;
};

// Exclusive offsets of the partition's tile left counts (at most
// kPlanScanTiles of them; more come with their offsets in a.tile_off) into
// s_off: per thread a run of consecutive tiles.
template <int T>
__device__ void plan_tile_offsets(const PlanArgs &a, int32_t *s_off)
{
    __shared__ int32_t s_w[T / 64];
    constexpr int kPer = (kPlanScanTiles + T - 1) / T;
    const int64_t t0 = (int64_t)threadIdx.x * kPer;
    int32_t v[kPer], run = 0;
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
        v[j] = t0 + j < a.tiles ? a.tile_cnt[t0 + j] : 0;
        run += v[j];
    }
    int32_t tot;
    int32_t o = plan_block_scan<T>(run, s_w, &tot);
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
        if (t0 + j <= kPlanScanTiles) s_off[t0 + j] = o;
        o += v[j];
    }
    __syncthreads();
}

// plan_node of level node t with its left count: from the partition's tile
// prefixes when a.tile_cnt is set (the left flags before its last slot's
// tile and within it, less those before its first slot; recorded in the
// node for later readers), else the node's own.  One read of the node.
__device__ inline PlanNode plan_node_counted(const PlanArgs &a, DevNode *__restrict__ nodes, int32_t t,
                                             const int32_t *s_off)
{
    const EvalNode e = a.cur[t];
    DevNode &d = nodes[e.heap];
    PlanNode x;
    x.p = e.heap;
    x.slot = e.slot;
    x.split = d.split;
    x.begin = d.begin;
    int64_t nl = d.nleft;
    if (a.tile_cnt) {
        nl = 0;
        if (d.end > d.begin) {
            const long long ob = a.tile_off ? a.tile_off[d.tile_b] : s_off[d.tile_b];
            const long long oe = a.tile_off ? a.tile_off[d.tile_e] : s_off[d.tile_e];
            nl = (oe + d.left_e) - (ob + d.left_b);
        }
        d.nleft = nl;
    }
    x.nl = nl;
    x.nr = d.end - d.begin - nl;
    x.lg = d.left_g;
    x.lh = d.left_h;
    x.rg = d.right_g;
    x.rh = d.right_h;
    x.pad0 = 0;
    return x;
}

template <int T>
__device__ void plan_level_block(DevNode *__restrict__ nodes, const PlanArgs &a)
{
    __shared__ int32_t lds16[T / 64];
    __shared__ unsigned long long red_rows[T / 64];
    __shared__ int32_t red_nodes[T / 64];
    // one pass's nodes: first work item (and the pass's end), row segment
    __shared__ int32_t s_kp[T + 1];
    __shared__ long long s_sb[T], s_se[T];
    __shared__ int32_t s_off[kPlanScanTiles + 1];
    const int32_t n_cur = *a.n_cur_d;
    if (a.tile_cnt && !a.tile_off) plan_tile_offsets<T>(a, s_off);
    // the children's segments and sums; the rows and nodes to build, for the
    // chunk size (a level of at most T nodes keeps each thread's node in
    // registers for the second pass; a thread handles the same nodes in
    // both, so a larger level's second pass reads the left counts its
    // thread recorded)
    PlanNode mine{};
    unsigned long long rb = 0;
    int32_t nbuild = 0;
    for (int32_t t = threadIdx.x; t < n_cur; t += T) {
        const PlanNode x = plan_node_counted(a, nodes, t, s_off);
        if (t < T) mine = x;
        if (!x.split) continue;
        DevNode &L = nodes[2 * x.p + 1];
        DevNode &Rn = nodes[2 * x.p + 2];
        L.present = 1;
        L.sum_g = x.lg;
        L.sum_h = x.lh;
        L.begin = x.begin;
        L.end = x.begin + x.nl;
        Rn.present = 1;
        Rn.sum_g = x.rg;
        Rn.sum_h = x.rh;
        Rn.begin = x.begin + x.nl;
        Rn.end = x.begin + x.nl + x.nr;
        rb += (unsigned long long)(x.nl <= x.nr ? x.nl : x.nr);
        ++nbuild;
    }
    if (a.lv.leaf) {
        __syncthreads();  // every child's record is written
        const int32_t eg = a.lv.e_dev[0], eh = a.lv.e_dev[1];
        for (int32_t i = threadIdx.x; i < a.lv.n_nodes; i += T)
            leaf_entry(nodes, i, eg, eh, a.lv.lambda, a.lv.eta, a.lv.leaf, a.lv.compact);
    }
    if (!a.plan) return;
    rb = wave_total(rb);
    nbuild = wave_total(nbuild);
    if ((threadIdx.x & 63) == 0) {
        red_rows[threadIdx.x >> 6] = rb;
        red_nodes[threadIdx.x >> 6] = nbuild;
    }
    __syncthreads();
    unsigned long long rows_total = 0;
    int32_t nodes_total = 0;
    for (int w = 0; w < T / 64; ++w) {
        rows_total += red_rows[w];
        nodes_total += red_nodes[w];
    }
    // room for the chunks of large nodes: what the node count leaves of the
    // target; a level of more than items / 2 nodes takes chunks of
    // rows_total / items rows (nodes smaller than the target's share would
    // otherwise take one chunk each and leave workgroup slots idle; up to
    // items + nodes_total work items)
    const int64_t items = a.items;
    const int64_t room = items - nodes_total > items / 2 ? items - nodes_total : items;
    int64_t chunk = ((int64_t)rows_total + room - 1) / room;
    chunk = chunk > kMinChunk ? chunk : kMinChunk;
    int32_t c_build = 0, c_part = 0;
    unsigned long long rows_built = 0;
    for (int32_t base = 0; base < n_cur; base += T) {
        const int32_t t = base + (int32_t)threadIdx.x;
        PlanNode x{};
        if (t < n_cur) x = n_cur <= T ? mine : plan_node(a.cur, nodes, t);
        const bool split = t < n_cur && x.split;
        int32_t nchunks = 0;
        if (split) {
            const int64_t ns = x.nl <= x.nr ? x.nl : x.nr;
            nchunks = (int32_t)(ns > 0 ? (ns + chunk - 1) / chunk : 1);
            rows_built += (unsigned long long)ns;
        }
        // one scan of both counts: the split flags in the low 16 bits (at
        // most T of them), the chunks above (at most items + T per pass)
        int32_t tot;
        const int32_t pre = plan_block_scan<T>((split ? 1 : 0) | (nchunks << 16), lds16, &tot);
        const int32_t tot_b = tot & 0xffff, tot_p = tot >> 16;
        const int32_t kb = (pre & 0xffff) + c_build;
        const int32_t kp = (pre >> 16) + c_part;
        if (split) {
            const int32_t sl = 2 * kb, sr = sl + 1;  // the children of split parents, in heap order
            a.next[sl] = {x.lg, x.lh, sl, 2 * x.p + 1};
            a.next[sr] = {x.rg, x.rh, sr, 2 * x.p + 2};
            nodes[2 * x.p + 1].slot = sl;
            nodes[2 * x.p + 2].slot = sr;
            const bool left_small = x.nl <= x.nr;
            const int64_t sb = left_small ? x.begin : x.begin + x.nl;
            const int64_t se = left_small ? x.begin + x.nl : x.begin + x.nl + x.nr;
            a.red[kb] = {left_small ? sl : sr, kp, nchunks, x.slot, left_small ? sr : sl, 0};
            s_sb[threadIdx.x] = sb;
            s_se[threadIdx.x] = se;
        }
        s_kp[threadIdx.x] = kp;
        if (threadIdx.x == T - 1) s_kp[T] = c_part + tot_p;
        __syncthreads();
        // the pass's work items, written by all threads: item e belongs to
        // the last node whose first item is <= e (nodes without items have
        // the next node's first item)
        for (int32_t e = c_part + (int32_t)threadIdx.x; e < c_part + tot_p; e += T) {
            int32_t lo = 0, hi = T;  // s_kp[lo] <= e < s_kp[hi]
            while (hi - lo > 1) {
                const int32_t mid = (lo + hi) >> 1;
                if (s_kp[mid] <= e)
                    lo = mid;
                else
                    hi = mid;
            }
            const int64_t b = s_sb[lo] + (int64_t)(e - s_kp[lo]) * chunk;
            a.work[e] = {b, b + chunk < s_se[lo] ? b + chunk : s_se[lo], e, 0};
        }
        __syncthreads();
        c_build += tot_b;
        c_part += tot_p;
    }
    rows_built = wave_total(rows_built);
    if ((threadIdx.x & 63) == 0 && rows_built) atomicAdd(&a.stat[0], rows_built);
    if (threadIdx.x == 0) {
        *a.n_next_d = 2 * c_build;
        *a.n_red_d = c_build;
        *a.n_work_d = c_part;
        atomicAdd(&a.stat[1], (unsigned long long)c_build);
    }
}

}  // namespace gbt
