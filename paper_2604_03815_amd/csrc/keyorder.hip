// Key order and superblock bounds for the score+select kernel.
//
// Every key the select kernel skips must provably score no more than the
// query's threshold.  Keys are grouped into superblocks of 256 (kSuperTiles
// tiles), each with a ball that contains all of its keys: a center c (the
// mean, rounded to bf16) and a radius R >= |k - c| with margins that cover
// the rounding of the scores (see sb_bounds_kernel).  For a query q every
// key of the superblock then scores at most q.c + |q| R, and a superblock
// whose bound does not beat any of a wave's thresholds is skipped.
//
// The bounds are tight when each superblock is small in every direction.
// The keys are therefore stored, per head, in the leaf order of a balanced
// binary space-partitioning tree: each node splits its keys at the median of
// their projections on the node's principal axis (estimated by power
// iteration on an evenly spaced sample of the node), with the left part
// rounded up to a whole number of superblocks, down to nodes of at most 256
// keys.  Every leaf is then exactly one superblock.  The tree is built level
// by level; a level's split is an exact selection of the left part by a
// two-pass radix select on a 16-bit quantisation of the projections (keys
// with the split value are assigned to the two sides by ticket).  The order
// only decides which tiles the select kernel visits together: it records
// each candidate by its original key index, so the result does not depend
// on it.
#include <utility>

#include "kmip_device.h"
#include "kmip_internal.h"

namespace kmip {
namespace {

constexpr int SBK = kSuperTiles * 32;  // keys per superblock
static_assert(SBK == 256, "one thread per key of a superblock");
constexpr int kSample = 64;            // keys sampled per node for its axis
constexpr int kPowerIters = 5;

// Per-node working data of one level, [H][width]:
//   f: mean[d], axis[d], lo, inv_step (projection p maps to
//      clamp((p - lo) * inv_step) in 0 .. 65535)
//   h: hist1[256], hist2[256], then the counters and split search results
constexpr int kLeftCursor = 512;  // and kLeftCursor + 1: the right side's
constexpr int kTieTicket = 514;
constexpr int kHighByte = 515;
constexpr int kSplitValue = 516;
constexpr int kTiesLeft = 517;
constexpr int kNodeInts = 520;

// Size of the left part of a node of n > SBK keys: half, rounded up to whole
// superblocks, and at least one key on the right.
__host__ __device__ __forceinline__ int split_left(int n) {
    const int half = (n + 1) / 2;
    const int nl = (half + SBK - 1) / SBK * SBK;
    return nl < n - 1 ? nl : n - 1;
}

// Node of level lev (root: 0) that holds position p: its first position lo,
// size n and index among the level's nodes.  False when p lies in a leaf of
// an earlier level (no longer split).
__device__ __forceinline__ bool node_of(int p, int N, int lev, int& lo, int& n, int& idx) {
    lo = 0;
    n = N;
    idx = 0;
    for (int l = 0; l < lev; ++l) {
        if (n <= SBK) return false;
        const int nl = split_left(n);
        if (p < lo + nl) {
            n = nl;
            idx = 2 * idx;
        } else {
            lo += nl;
            n -= nl;
            idx = 2 * idx + 1;
        }
    }
    return n > SBK;
}

// Node idx of level lev by its path (bit lev-1-l of idx picks the side at
// level l).  False when the path ends in a leaf before level lev.
__device__ __forceinline__ bool node_by_index(int idx, int N, int lev, int& lo, int& n) {
    lo = 0;
    n = N;
    for (int l = 0; l < lev; ++l) {
        if (n <= SBK) return false;
        const int nl = split_left(n);
        if (((idx >> (lev - 1 - l)) & 1) == 0) {
            n = nl;
        } else {
            lo += nl;
            n -= nl;
        }
    }
    return n > SBK;
}

// Reductions over the 64 lanes of a wave (all active), returning the same
// value to every lane: an inclusive scan within each row of 16 lanes by DPP
// row shifts (lanes shifted in from outside the row contribute `fill`, the
// operation's identity), then the four row totals (lanes 15, 31, 47, 63)
// read as scalars.  The chain is four dependent DPP steps, far shorter than
// a butterfly through the LDS crossbar.
template <int CTRL>
__device__ __forceinline__ float dpp_row_shr(float v, float fill) {
    return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(fill), __float_as_int(v), CTRL, 0xf,
                                                      0xf, false));
}

__device__ __forceinline__ float lane_f(float v, int lane) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}

__device__ __forceinline__ float wave_sum(float v) {
    v += dpp_row_shr<0x111>(v, 0.0f);
    v += dpp_row_shr<0x112>(v, 0.0f);
    v += dpp_row_shr<0x114>(v, 0.0f);
    v += dpp_row_shr<0x118>(v, 0.0f);
    return (lane_f(v, 15) + lane_f(v, 31)) + (lane_f(v, 47) + lane_f(v, 63));
}

__device__ __forceinline__ float wave_max(float v) {
    v = fmaxf(v, dpp_row_shr<0x111>(v, -INFINITY));
    v = fmaxf(v, dpp_row_shr<0x112>(v, -INFINITY));
    v = fmaxf(v, dpp_row_shr<0x114>(v, -INFINITY));
    v = fmaxf(v, dpp_row_shr<0x118>(v, -INFINITY));
    return fmaxf(fmaxf(lane_f(v, 15), lane_f(v, 31)), fmaxf(lane_f(v, 47), lane_f(v, 63)));
}

__device__ __forceinline__ float wave_min(float v) {
    v = fminf(v, dpp_row_shr<0x111>(v, INFINITY));
    v = fminf(v, dpp_row_shr<0x112>(v, INFINITY));
    v = fminf(v, dpp_row_shr<0x114>(v, INFINITY));
    v = fminf(v, dpp_row_shr<0x118>(v, INFINITY));
    return fminf(fminf(lane_f(v, 15), lane_f(v, 31)), fminf(lane_f(v, 47), lane_f(v, 63)));
}

// One wave: the mean and principal axis of the S <= 64 sample rows x held by
// the active lanes (power iteration from the sample farthest from the mean),
// and the quantisation range of the sample's projections.  The lane with
// `writer` set stores the node record nf: mean[D], axis[D], qlo, qinv (codes
// map a projection p to clamp((p - qlo) * qinv) in 0 .. 65535).  x comes
// back mean-centred.
template <int D>
__device__ __forceinline__ void sample_axis(float (&x)[D], bool act, int S, bool writer,
                                            float* __restrict__ nf) {
    const float inv_s = 1.0f / (float)S;
    // static indices keep the arrays in registers
#pragma unroll
    for (int i = 0; i < D; ++i) {
        const float mu = wave_sum(x[i]) * inv_s;
        if (writer) nf[i] = mu;
        x[i] = act ? x[i] - mu : 0.0f;
    }
    float dd = 0.0f;
#pragma unroll
    for (int i = 0; i < D; ++i) dd = fmaf(x[i], x[i], dd);
    const float m = wave_max(dd);
    const int far = (int)__builtin_ctzll(__builtin_amdgcn_ballot_w64(dd == m));
    float axis[D];
#pragma unroll
    for (int i = 0; i < D; ++i) axis[i] = __shfl(x[i], far);
    // power iteration: axis <- sum_s (x_s . axis) x_s, normalised
    for (int it = 0; it < kPowerIters; ++it) {
        float nn = 0.0f;
#pragma unroll
        for (int i = 0; i < D; ++i) nn = fmaf(axis[i], axis[i], nn);
        const float inv = nn > 0.0f ? rsqrtf(nn) : 0.0f;
        float pr = 0.0f;
#pragma unroll
        for (int i = 0; i < D; ++i) pr = fmaf(x[i], axis[i] * inv, pr);
#pragma unroll
        for (int i = 0; i < D; ++i) axis[i] = wave_sum(pr * x[i]);
    }
    float nn = 0.0f;
#pragma unroll
    for (int i = 0; i < D; ++i) nn = fmaf(axis[i], axis[i], nn);
    if (nn > 0.0f) {
        const float inv = rsqrtf(nn);
#pragma unroll
        for (int i = 0; i < D; ++i) axis[i] *= inv;
    } else {
#pragma unroll
        for (int i = 0; i < D; ++i) axis[i] = i == 0 ? 1.0f : 0.0f;
    }
    float pr = 0.0f;
#pragma unroll
    for (int i = 0; i < D; ++i) pr = fmaf(x[i], axis[i], pr);
    const float pmin = wave_min(act ? pr : INFINITY), pmax = wave_max(act ? pr : -INFINITY);
    if (writer) {
#pragma unroll
        for (int i = 0; i < D; ++i) nf[D + i] = axis[i];
        // the mean-centred projection of the sample, widened a little so that
        // most keys fall inside the quantised range
        const float span = pmax - pmin;
        nf[2 * D] = pmin - 0.0625f * span;
        nf[2 * D + 1] = span > 0.0f ? 65535.0f / (1.125f * span) : 0.0f;
    }
}

// Level lev, one wave per node: the node's mean and principal axis from an
// evenly spaced sample of its keys, the quantisation range, and zeroed
// histograms and counters.
template <int D>
__global__ __launch_bounds__(64) void tree_axis_kernel(const uint16_t* __restrict__ kp, int32_t N,
                                                       int32_t H, int32_t lev, int32_t width,
                                                       float* __restrict__ nodef,
                                                       int32_t* __restrict__ nodeh) {
    const int idx = blockIdx.x;
    const int h = blockIdx.y;
    const int t = threadIdx.x;
    int lo, n;
    if (!node_by_index(idx, N, lev, lo, n)) return;
    int32_t* nh = nodeh + ((size_t)h * width + idx) * kNodeInts;
    for (int e = t; e < kNodeInts; e += 64) nh[e] = 0;
    const int S = n < kSample ? n : kSample;
    const bool act = t < S;
    float x[D];
    if (act) {
        const int p = lo + (int)(((int64_t)(2 * t + 1) * n) / (2 * S));
        load_row_f32<D>(x, kp + ((size_t)h * N + p) * D);
    } else {
#pragma unroll
        for (int i = 0; i < D; ++i) x[i] = 0.0f;
    }
    sample_axis<D>(x, act, S, t == 0, nodef + ((size_t)h * width + idx) * (2 * D + 2));
}

template <int D>
__device__ __forceinline__ uint32_t quantise(const float* __restrict__ nf, const float (&x)[D]) {
    float pr = 0.0f;
#pragma unroll
    for (int i = 0; i < D; ++i) pr = fmaf(x[i] - nf[i], nf[D + i], pr);
    const float u = (pr - nf[2 * D]) * nf[2 * D + 1];
    return (uint32_t)fminf(fmaxf(u, 0.0f), 65535.0f);
}

// The per-position level kernels give each block kBlockPos consecutive
// positions, kPerThread per thread in rounds of 256 (so that the lanes of a
// wave take consecutive positions, mostly of one node).  A block adds the
// histogram counts of the node that holds its first position in LDS and
// flushes them once: at the top levels, where all positions fall into few
// nodes, that keeps the global atomics on one node's 256 bins few.
constexpr int kPerThread = 8;
constexpr int kBlockPos = 256 * kPerThread;

// Adds 1 to *addr for every active lane and returns the lane's rank among
// the lanes of its wave with the same address: one atomic per distinct
// address in the wave.
__device__ __forceinline__ int wave_ticket(int32_t* addr, bool active) {
    const int lane = threadIdx.x & 63;
    const uint64_t below = (1ull << lane) - 1ull;
    int rank = 0;
    uint64_t todo = __builtin_amdgcn_ballot_w64(active);
    while (todo != 0ull) {
        const int leader = (int)__builtin_ctzll(todo);
        const uint64_t a = reinterpret_cast<uint64_t>(addr);
        const uint64_t la = (uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)a, leader) |
                            ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(a >> 32), leader) << 32);
        const bool mine = active && a == la;
        const uint64_t same = __builtin_amdgcn_ballot_w64(mine);
        int base = 0;
        if (lane == leader) base = atomicAdd(reinterpret_cast<int32_t*>(la), (int)__builtin_popcountll(same));
        base = __builtin_amdgcn_readlane(base, leader);
        if (mine) rank = base + (int)__builtin_popcountll(same & below);
        todo &= ~same;
    }
    return rank;
}

// Level lev: the 16-bit projection code of the key at each position of a
// split node, and the histogram of its high byte per node.
template <int D>
__global__ __launch_bounds__(256) void tree_project_kernel(const uint16_t* __restrict__ kp, int32_t N,
                                                           int32_t H, int32_t lev, int32_t width,
                                                           const float* __restrict__ nodef,
                                                           int32_t* __restrict__ nodeh,
                                                           uint16_t* __restrict__ code) {
    __shared__ int32_t lh[256];
    const int h = blockIdx.y;
    const int t = threadIdx.x;
    const int base = blockIdx.x * kBlockPos;
    int lo0, n0, idx0;
    const bool agg = node_of(base, N, lev, lo0, n0, idx0);
    lh[t] = 0;
    __syncthreads();
    for (int i = 0; i < kPerThread; ++i) {
        const int p = base + i * 256 + t;
        int lo, n, idx;
        if (p >= N || !node_of(p, N, lev, lo, n, idx)) continue;
        float x[D];
        load_row_f32<D>(x, kp + ((size_t)h * N + p) * D);
        const uint32_t q = quantise<D>(nodef + ((size_t)h * width + idx) * (2 * D + 2), x);
        code[(size_t)h * N + p] = (uint16_t)q;
        if (agg && idx == idx0)
            atomicAdd(&lh[q >> 8], 1);
        else
            atomicAdd(&nodeh[((size_t)h * width + idx) * kNodeInts + (q >> 8)], 1);
    }
    __syncthreads();
    if (agg && lh[t] != 0) atomicAdd(&nodeh[((size_t)h * width + idx0) * kNodeInts + t], lh[t]);
}

// Level lev, one block per split node: the split search on one of its
// histograms.  Pass 0 finds the bin of the high byte that holds the
// node's nl-th smallest code (0-based: the first position of the right
// side); pass 1 finds the low byte within that bin.  Afterwards
// kSplitValue holds the code v at which the node splits and kTiesLeft how
// many keys with code v go left (the keys with a smaller code all do).
__global__ __launch_bounds__(256) void tree_find_kernel(int32_t N, int32_t lev, int32_t width,
                                                        int32_t pass, int32_t* __restrict__ nodeh) {
    __shared__ int32_t sc[256];
    const int idx = blockIdx.x;
    const int h = blockIdx.y;
    const int t = threadIdx.x;
    int lo, n;
    if (!node_by_index(idx, N, lev, lo, n)) return;
    int32_t* nh = nodeh + ((size_t)h * width + idx) * kNodeInts;
    const int target = pass == 0 ? split_left(n) : nh[kTiesLeft];
    const int v = nh[pass * 256 + t];
    sc[t] = v;
    __syncthreads();
    for (int off = 1; off < 256; off <<= 1) {
        const int add = t >= off ? sc[t - off] : 0;
        __syncthreads();
        sc[t] += add;
        __syncthreads();
    }
    const int incl = sc[t], excl = incl - v;
    if (target >= excl && target < incl) {
        if (pass == 0) {
            nh[kHighByte] = t;
            nh[kTiesLeft] = target - excl;
        } else {
            nh[kSplitValue] = (nh[kHighByte] << 8) | t;
            nh[kTiesLeft] = target - excl;
        }
    }
}

// Level lev: histogram of the low byte of the codes whose high byte is the
// split bin of their node.
__global__ __launch_bounds__(256) void tree_hist2_kernel(int32_t N, int32_t lev, int32_t width,
                                                         int32_t* __restrict__ nodeh,
                                                         const uint16_t* __restrict__ code) {
    __shared__ int32_t lh[256];
    const int h = blockIdx.y;
    const int t = threadIdx.x;
    const int base = blockIdx.x * kBlockPos;
    int lo0, n0, idx0;
    const bool agg = node_of(base, N, lev, lo0, n0, idx0);
    const int b0 = agg ? nodeh[((size_t)h * width + idx0) * kNodeInts + kHighByte] : -1;
    lh[t] = 0;
    __syncthreads();
    for (int i = 0; i < kPerThread; ++i) {
        const int p = base + i * 256 + t;
        int lo, n, idx;
        if (p >= N || !node_of(p, N, lev, lo, n, idx)) continue;
        const uint32_t q = code[(size_t)h * N + p];
        int32_t* nh = nodeh + ((size_t)h * width + idx) * kNodeInts;
        const bool own = agg && idx == idx0;
        if ((int)(q >> 8) != (own ? b0 : nh[kHighByte])) continue;
        if (own)
            atomicAdd(&lh[q & 255u], 1);
        else
            atomicAdd(&nh[256 + (q & 255u)], 1);
    }
    __syncthreads();
    if (agg && lh[t] != 0) atomicAdd(&nodeh[((size_t)h * width + idx0) * kNodeInts + 256 + t], lh[t]);
}

// Level lev: every position of a split node moves to its side.  The left
// side takes the keys whose code is below the split value and, by ticket,
// as many keys with the split value as it still needs.  Positions in leaves
// keep their key.  A block's positions take their ranks from LDS counters,
// one per (node, side), and the block reserves its places in each node with
// one global atomic: split nodes hold more than SBK positions, so the slot
// (lo - base) / (SBK + 1) + 1 of a node starting inside the block (0 for the
// one it starts in) tells its nodes apart.
constexpr int kSlots = kBlockPos / (SBK + 1) + 2;

// The key rows of the head-major copy move with their keys.
template <int D>
__global__ __launch_bounds__(256) void tree_scatter_kernel(int32_t N, int32_t lev, int32_t width,
                                                           int32_t* __restrict__ nodeh,
                                                           const uint16_t* __restrict__ code,
                                                           const int32_t* __restrict__ perm_in,
                                                           int32_t* __restrict__ perm_out,
                                                           const uint16_t* __restrict__ kp_in,
                                                           uint16_t* __restrict__ kp_out) {
    __shared__ int32_t cnt[kSlots][2];
    __shared__ int32_t sidx[kSlots];
    const int h = blockIdx.y;
    const int t = threadIdx.x;
    const int base = blockIdx.x * kBlockPos;
    if (t < 2 * kSlots) cnt[t >> 1][t & 1] = 0;
    __syncthreads();
    int dst[kPerThread], slot[kPerThread], side[kPerThread], rank[kPerThread];
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) {
        const int p = base + i * 256 + t;
        int lo = 0, n = 0, idx = 0;
        const bool split = p < N && node_of(p, N, lev, lo, n, idx);
        int32_t* nh = nodeh + ((size_t)h * width + (split ? idx : 0)) * kNodeInts;
        const int q = split ? (int)code[(size_t)h * N + p] : 0;
        const int v = split ? nh[kSplitValue] : 0;
        const bool tie = split && q == v;
        // every lane takes part in the ticket, active or not
        const int ticket = wave_ticket(nh + kTieTicket, tie);
        side[i] = q < v ? 0 : (q > v ? 1 : (ticket < nh[kTiesLeft] ? 0 : 1));
        slot[i] = -1;
        dst[i] = p;
        if (split) {
            slot[i] = lo < base ? 0 : (lo - base) / (SBK + 1) + 1;
            sidx[slot[i]] = idx;
            rank[i] = atomicAdd(&cnt[slot[i]][side[i]], 1);
            dst[i] = lo + (side[i] == 0 ? 0 : split_left(n)) + rank[i];
        }
    }
    __syncthreads();
    if (t < 2 * kSlots) {
        const int s = t >> 1, sd = t & 1;
        const int c = cnt[s][sd];
        if (c != 0) cnt[s][sd] = atomicAdd(&nodeh[((size_t)h * width + sidx[s]) * kNodeInts + kLeftCursor + sd], c);
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) {
        const int p = base + i * 256 + t;
        if (p >= N) continue;
        const int32_t key = perm_in[(size_t)h * N + p];
        const size_t to = (size_t)h * N + dst[i] + (slot[i] >= 0 ? cnt[slot[i]][side[i]] : 0);
        perm_out[to] = key;
        const uint4* src = reinterpret_cast<const uint4*>(kp_in + ((size_t)h * N + p) * D);
        uint4* out = reinterpret_cast<uint4*>(kp_out + to * D);
#pragma unroll
        for (int c = 0; c < D / 8; ++c) out[c] = src[c];
    }
}

// The bottom levels in one launch.  Once every split node of level lev0
// holds at most kLocalRows(D) keys (their rows fill 128 KB of LDS), one
// block per node loads the node's rows and runs all remaining levels in LDS:
// the same sample axis, quantisation and exact two-pass split as the
// per-level kernels, with the keys of the split value assigned to the left
// side in position order.  Only a permutation of the node's positions moves
// between levels; at the end the rows and key ids are written back in their
// final order, in place (blocks own disjoint position ranges).
//
// Sub-nodes: a node of n <= 256 MS keys (MS a power of two) has every
// sub-node at depth j at most 256 MS / 2^j keys (the left part rounds half
// up to whole superblocks, which keeps that bound), so sub-nodes that are
// still split (more than 256 keys) occur only at depths with 2^j <= MS / 2,
// and their path index is below MS.
template <int D>
constexpr int kLocalRows = 65536 / D;

template <int D>
__global__ __launch_bounds__(512) void tree_local_kernel(int32_t N, int32_t lev0,
                                                         uint16_t* __restrict__ kp,
                                                         int32_t* __restrict__ perm) {
    constexpr int NL = kLocalRows<D>;
    constexpr int NT = 512;
    constexpr int NW = NT / 64;
    constexpr int PT = NL / NT;   // positions per thread, consecutive
    constexpr int MS = NL / SBK;  // bound on the index of a split sub-node
    constexpr int RW = D / 8;     // uint4 per row
    __shared__ uint4 rows[NL * RW];
    __shared__ uint16_t ord[2][NL];      // ord[.][position] = row of the node in LDS
    __shared__ uint32_t hist[MS][128];   // two 16-bit bins per word
    __shared__ float subf[MS][2 * D + 2];
    __shared__ int32_t subi[MS][4];      // split value, ties to the left, high byte, prefix base
    __shared__ uint32_t wtot[NW];
    const int h = blockIdx.y;
    const int t = threadIdx.x;
    const int wave = t >> 6, lane = t & 63;
    int lo, n;
    if (!node_by_index(blockIdx.x, N, lev0, lo, n)) return;
    if (n > NL) return;   // the host starts at a level where no node is larger
    const uint4* src = reinterpret_cast<const uint4*>(kp + ((size_t)h * N + lo) * D);
    // eight loads in flight per thread before their LDS stores
    static_assert(NL * RW % (8 * NT) == 0, "whole rounds of eight");
    for (int e0 = 0; e0 < NL * RW; e0 += 8 * NT) {
        uint4 buf[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int e = e0 + u * NT + t;
            if (e < n * RW) buf[u] = src[e];
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int e = e0 + u * NT + t;
            if (e < n * RW) rows[e] = buf[u];
        }
    }
    for (int p = t; p < n; p += NT) ord[0][p] = (uint16_t)p;
    __syncthreads();
    int cb = 0;
    for (int j = 0;; ++j) {
        // the left-most sub-node is the largest of its depth
        int big = n;
        for (int l = 0; l < j && big > SBK; ++l) big = split_left(big);
        if (big <= SBK) break;
        // sample axis of every split sub-node, one wave each; clear its histogram
        for (int sidx = wave; sidx < MS && sidx < (1 << j); sidx += NW) {
            int slo, sn;
            if (!node_by_index(sidx, n, j, slo, sn)) continue;
            float x[D];
            const int p = slo + (int)(((int64_t)(2 * lane + 1) * sn) / (2 * kSample));
            load_row_f32<D>(x, reinterpret_cast<const uint16_t*>(&rows[(int)ord[cb][p] * RW]));
            sample_axis<D>(x, true, kSample, lane == 0, subf[sidx]);
            hist[sidx][2 * lane] = 0u;
            hist[sidx][2 * lane + 1] = 0u;
        }
        __syncthreads();
        // codes and the high-byte histograms
        int code[PT], sid[PT], sblo[PT], sbn[PT];
#pragma unroll
        for (int i = 0; i < PT; ++i) {
            const int p = t * PT + i;
            int slo = 0, sn = 0, sidx = -1;
            code[i] = 0;
            if (p < n && node_of(p, n, j, slo, sn, sidx) && sidx < MS) {
                float x[D];
                load_row_f32<D>(x, reinterpret_cast<const uint16_t*>(&rows[(int)ord[cb][p] * RW]));
                code[i] = (int)quantise<D>(subf[sidx], x);
                atomicAdd(&hist[sidx][code[i] >> 9], 1u << (((code[i] >> 8) & 1) << 4));
            } else {
                sidx = -1;
            }
            sid[i] = sidx;
            sblo[i] = slo;
            sbn[i] = sn;
        }
        __syncthreads();
        // two passes of the split search, one wave per split sub-node: the
        // bin that holds the target rank, then the value within that bin
        for (int pass = 0; pass < 2; ++pass) {
            for (int sidx = wave; sidx < MS && sidx < (1 << j); sidx += NW) {
                int slo, sn;
                if (!node_by_index(sidx, n, j, slo, sn)) continue;
                const int target = pass == 0 ? split_left(sn) : subi[sidx][1];
                const uint32_t w0 = hist[sidx][2 * lane], w1 = hist[sidx][2 * lane + 1];
                const int c[4] = {(int)(w0 & 0xFFFFu), (int)(w0 >> 16), (int)(w1 & 0xFFFFu), (int)(w1 >> 16)};
                const int mine = c[0] + c[1] + c[2] + c[3];
                int incl = mine;
#pragma unroll
                for (int off = 1; off < 64; off <<= 1) {
                    const int o = __shfl_up(incl, off);
                    if (lane >= off) incl += o;
                }
                int below = incl - mine;
                if (target >= below && target < incl) {
                    int b = 0;
                    if (target >= below + c[0]) {
                        below += c[0];
                        b = 1;
                        if (target >= below + c[1]) {
                            below += c[1];
                            b = 2;
                            if (target >= below + c[2]) {
                                below += c[2];
                                b = 3;
                            }
                        }
                    }
                    const int bin = 4 * lane + b;
                    if (pass == 0) {
                        subi[sidx][2] = bin;
                    } else {
                        subi[sidx][0] = (subi[sidx][2] << 8) | bin;
                    }
                    subi[sidx][1] = target - below;
                }
                hist[sidx][2 * lane] = 0u;
                hist[sidx][2 * lane + 1] = 0u;
            }
            __syncthreads();
            if (pass == 0) {
#pragma unroll
                for (int i = 0; i < PT; ++i) {
                    if (sid[i] >= 0 && (code[i] >> 8) == subi[sid[i]][2])
                        atomicAdd(&hist[sid[i]][(code[i] & 255) >> 1], 1u << ((code[i] & 1) << 4));
                }
                __syncthreads();
            }
        }
        // partition: a block-wide scan of (code < v) + (code == v) << 16
        uint32_t pre[PT];
        uint32_t tot = 0u;
#pragma unroll
        for (int i = 0; i < PT; ++i) {
            pre[i] = tot;
            if (sid[i] >= 0) {
                const int v = subi[sid[i]][0];
                tot += code[i] < v ? 1u : (code[i] == v ? 0x10000u : 0u);
            }
        }
        uint32_t incl = tot;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const uint32_t o = __shfl_up(incl, off);
            if (lane >= off) incl += o;
        }
        if (lane == 63) wtot[wave] = incl;
        __syncthreads();
        uint32_t base = incl - tot;
        for (int w = 0; w < wave; ++w) base += wtot[w];
#pragma unroll
        for (int i = 0; i < PT; ++i) {
            if (sid[i] >= 0 && t * PT + i == sblo[i]) subi[sid[i]][3] = (int)(base + pre[i]);
        }
        __syncthreads();
#pragma unroll
        for (int i = 0; i < PT; ++i) {
            const int p = t * PT + i;
            if (p >= n) continue;
            int dst = p;
            if (sid[i] >= 0) {
                const int s2 = sid[i];
                const uint32_t rel = base + pre[i] - (uint32_t)subi[s2][3];
                const int ltb = (int)(rel & 0xFFFFu), tieb = (int)(rel >> 16);
                const int tl = subi[s2][1];
                const int v = subi[s2][0];
                const int leftb = ltb + (tieb < tl ? tieb : tl);
                const bool left = code[i] < v || (code[i] == v && tieb < tl);
                dst = left ? sblo[i] + leftb : sblo[i] + split_left(sbn[i]) + (p - sblo[i] - leftb);
            }
            ord[cb ^ 1][dst] = ord[cb][p];
        }
        __syncthreads();
        cb ^= 1;
    }
    // write back: read every key id first, then overwrite the node's range
    int32_t* pk = perm + (size_t)h * N + lo;
    int32_t key[PT];
#pragma unroll
    for (int i = 0; i < PT; ++i) {
        const int p = t + i * NT;
        key[i] = p < n ? pk[(int)ord[cb][p]] : 0;
    }
    __syncthreads();
    uint4* dstr = reinterpret_cast<uint4*>(kp + ((size_t)h * N + lo) * D);
#pragma unroll
    for (int i = 0; i < PT; ++i) {
        const int p = t + i * NT;
        if (p >= n) continue;
        pk[p] = key[i];
        const int r = (int)ord[cb][p];
#pragma unroll
        for (int c = 0; c < RW; ++c) dstr[p * RW + c] = rows[r * RW + c];
    }
}

// perm[h][p] = p and the head-major copy kp[h][p] = K row (p, h).
template <int D>
__global__ __launch_bounds__(256) void tree_init_kernel(const uint16_t* __restrict__ K, int32_t N, int32_t H,
                                                        int32_t* __restrict__ perm, uint16_t* __restrict__ kp) {
    const int p = blockIdx.x * 256 + threadIdx.x;
    const int h = blockIdx.y;
    if (p >= N) return;
    perm[(size_t)h * N + p] = p;
    const uint4* src = reinterpret_cast<const uint4*>(K + ((size_t)p * H + h) * D);
    uint4* dst = reinterpret_cast<uint4*>(kp + ((size_t)h * N + p) * D);
#pragma unroll
    for (int c = 0; c < D / 8; ++c) dst[c] = src[c];
}

// bf16 bits of x rounded to nearest even (finite x).
__device__ __forceinline__ uint16_t bf16_rne(float x) {
    const uint32_t b = __float_as_uint(x);
    return (uint16_t)((b + 0x7FFFu + ((b >> 16) & 1u)) >> 16);
}

// bf16 bits of the smallest bf16 >= x, for finite x >= 0.
__device__ __forceinline__ uint16_t bf16_up(float x) {
    const uint32_t b = __float_as_uint(x);
    return (uint16_t)((b >> 16) + ((b & 0xFFFFu) != 0u ? 1u : 0u));
}

// One block per superblock s of head h (its 256 keys are positions 256 s ..
// of the order; positions >= N are absent).  Writes the superblock's row of
// the bound tiles: tile s / 32, row s % 32, in the key-tile operand layout
// with NC + 1 chunks of 16 dims.  Chunks 0 .. NC-1 hold c, the mean of the
// keys rounded to bf16; chunk NC holds R_up in its first dim and zeros
// elsewhere.  A query's bound tile row q is then (q, |q|_up, 0 ..) . (c,
// R_up, 0 ..), formed by the same MFMA as the scores.
//
// Why the bound holds for the MFMA scores: every key k of the superblock
// has q.k = q.c + q.(k - c) <= q.c + |q| r with r = max |k - c|.  The radius
// r is computed in fp32 from bf16 data (relative error below (D/2 + 2)
// 2^-24), the MFMA's fp32 sums of D + 16 products err by less than about
// (D + 16) 2^-24 (|q||c| + |q||k| + |q| R) on both the score and the bound,
// and |k| <= |c| + r.  R = r (1 + 2^-12) + |c| 2^-12 exceeds r by far more
// than all of these together for D <= 64, and rounding R and |q| up to bf16
// only raises the bound further.  An empty superblock gets c = 0, R = 0;
// the select kernel never scans superblocks past the last one anyway.
template <int D>
__global__ __launch_bounds__(256) void sb_bounds_kernel(const uint16_t* __restrict__ kp, int32_t N,
                                                        int32_t H, int32_t ctiles,
                                                        uint16_t* __restrict__ bounds) {
    constexpr int NC = D / 16;
    __shared__ float part[4][D];
    __shared__ float cen[D];
    __shared__ float rpart[4];
    const int s = blockIdx.x;
    const int h = blockIdx.y;
    const int t = threadIdx.x;
    const int wave = t >> 6;
    const int64_t pos = (int64_t)s * SBK + t;
    const bool valid = pos < N;
    float x[D];
    if (valid) {
        load_row_f32<D>(x, kp + ((size_t)h * N + pos) * D);
    } else {
#pragma unroll
        for (int i = 0; i < D; ++i) x[i] = 0.0f;
    }
#pragma unroll
    for (int i = 0; i < D; ++i) {
        const float v = wave_sum(x[i]);
        if ((t & 63) == 0) part[wave][i] = v;
    }
    __syncthreads();
    const int64_t left = (int64_t)N - (int64_t)s * SBK;
    const int count = left <= 0 ? 0 : (left >= SBK ? SBK : (int)left);
    const int row = s & 31;
    uint16_t* tile = bounds + (((size_t)h * ctiles + (s >> 5)) * (NC + 1)) * 64 * 8;
    if (t < D) {
        const float sum = (part[0][t] + part[1][t]) + (part[2][t] + part[3][t]);
        const uint16_t cb = count > 0 ? bf16_rne(sum / (float)count) : (uint16_t)0;
        cen[t] = bf16_bits_to_f32(cb);
        tile[((t >> 4) * 64 + row + 32 * ((t >> 3) & 1)) * 8 + (t & 7)] = cb;
    }
    __syncthreads();
    float d2 = 0.0f;
    if (valid) {
#pragma unroll
        for (int i = 0; i < D; ++i) {
            const float e = x[i] - cen[i];
            d2 = fmaf(e, e, d2);
        }
    }
    const float m = wave_max(d2);
    if ((t & 63) == 0) rpart[wave] = m;
    __syncthreads();
    if (t >= D && t < D + 16) {
        const int j = t - D;
        uint16_t v = 0;
        if (j == 0 && count > 0) {
            float cn2 = 0.0f;
            for (int i = 0; i < D; ++i) cn2 = fmaf(cen[i], cen[i], cn2);
            const float r = sqrtf(fmaxf(fmaxf(rpart[0], rpart[1]), fmaxf(rpart[2], rpart[3])));
            const float R = fmaf(r, 1.0f + 0x1p-12f, sqrtf(cn2) * 0x1p-12f);
            v = bf16_up(R);
        }
        tile[(NC * 64 + row + 32 * (j >> 3)) * 8 + (j & 7)] = v;
    }
}

// One block per window w of head h: the 64 superblocks 64 w .. 64 w + 63,
// positions 16384 w .. (positions >= N are absent).  Writes the window's row
// of the window tiles (tile w / 32, row w % 32, same layout as the bound
// tiles): the centre c, the mean of the window's keys rounded to bf16, and
// R_up = bf16_up(r (1 + 2^-12) + |c| 2^-12) with r = max |k - c| over the
// window, the construction of sb_bounds_kernel over 16384 keys instead of
// 256.  The margin argument given there does not depend on how many keys a
// ball holds, so q.c + |q|_up R_up bounds the MFMA score of every key of the
// window: a window whose bound beats no query's threshold holds no key that
// can pass the select kernel's filter.  An empty window gets c = 0, R = 0.
template <int D>
__global__ __launch_bounds__(256) void win_bounds_kernel(const uint16_t* __restrict__ kp, int32_t N,
                                                         int32_t H, int32_t wctiles,
                                                         uint16_t* __restrict__ wbounds) {
    constexpr int NC = D / 16;
    constexpr int WK = 64 * SBK;   // keys per window
    __shared__ float part[4][D];
    __shared__ float cen[D];
    __shared__ float rpart[4];
    const int w = blockIdx.x;
    const int h = blockIdx.y;
    const int t = threadIdx.x;
    const int wave = t >> 6;
    const int64_t p0 = (int64_t)w * WK;
    const int64_t p1 = p0 + WK < (int64_t)N ? p0 + WK : (int64_t)N;
    const int count = p1 > p0 ? (int)(p1 - p0) : 0;
    float sum[D];
#pragma unroll
    for (int i = 0; i < D; ++i) sum[i] = 0.0f;
    for (int64_t pos = p0 + t; pos < p1; pos += 256) {
        float x[D];
        load_row_f32<D>(x, kp + ((size_t)h * N + pos) * D);
#pragma unroll
        for (int i = 0; i < D; ++i) sum[i] += x[i];
    }
#pragma unroll
    for (int i = 0; i < D; ++i) {
        const float v = wave_sum(sum[i]);
        if ((t & 63) == 0) part[wave][i] = v;
    }
    __syncthreads();
    const int row = w & 31;
    uint16_t* tile = wbounds + (((size_t)h * wctiles + (w >> 5)) * (NC + 1)) * 64 * 8;
    if (t < D) {
        const float tot = (part[0][t] + part[1][t]) + (part[2][t] + part[3][t]);
        const uint16_t cb = count > 0 ? bf16_rne(tot / (float)count) : (uint16_t)0;
        cen[t] = bf16_bits_to_f32(cb);
        tile[((t >> 4) * 64 + row + 32 * ((t >> 3) & 1)) * 8 + (t & 7)] = cb;
    }
    __syncthreads();
    float d2 = 0.0f;
    for (int64_t pos = p0 + t; pos < p1; pos += 256) {
        float x[D];
        load_row_f32<D>(x, kp + ((size_t)h * N + pos) * D);
        float e2 = 0.0f;
#pragma unroll
        for (int i = 0; i < D; ++i) {
            const float e = x[i] - cen[i];
            e2 = fmaf(e, e, e2);
        }
        d2 = fmaxf(d2, e2);
    }
    const float m = wave_max(d2);
    if ((t & 63) == 0) rpart[wave] = m;
    __syncthreads();
    if (t >= D && t < D + 16) {
        const int j = t - D;
        uint16_t v = 0;
        if (j == 0 && count > 0) {
            float cn2 = 0.0f;
            for (int i = 0; i < D; ++i) cn2 = fmaf(cen[i], cen[i], cn2);
            const float r = sqrtf(fmaxf(fmaxf(rpart[0], rpart[1]), fmaxf(rpart[2], rpart[3])));
            const float R = fmaf(r, 1.0f + 0x1p-12f, sqrtf(cn2) * 0x1p-12f);
            v = bf16_up(R);
        }
        tile[(NC * 64 + row + 32 * (j >> 3)) * 8 + (j & 7)] = v;
    }
}

// Levels of splitting for N keys: nodes of level l are split while l <
// levels (the deepest split level has at most width nodes).
void tree_shape(int32_t N, int32_t& levels, int32_t& width) {
    const int32_t nsb = (N + SBK - 1) / SBK;
    levels = 0;
    while ((1 << levels) < nsb) ++levels;
    width = levels > 0 ? (1 << (levels - 1)) : 1;
}

// First level at which every split node fits tree_local_kernel (nl keys),
// or levels.  The left-most node of a level is its largest.
int32_t tree_local_level(int32_t N, int32_t levels, int32_t nl) {
    int32_t big = N;
    for (int32_t lev = 0; lev < levels; ++lev) {
        if (big <= nl) return lev;
        big = big > SBK ? split_left(big) : big;
    }
    return levels;
}

}  // namespace

int32_t key_order_ctiles(int32_t ntiles) {
    const int32_t nsb = (ntiles + kSuperTiles - 1) / kSuperTiles;
    return (nsb + 63) / 64 * 2;
}

int32_t key_order_wctiles(int32_t ctiles) {
    const int32_t nwin = ctiles / 2;   // one window per pair of bound tiles
    return (nwin + 63) / 64 * 2;
}

size_t key_order_workspace_bytes(int32_t N, int32_t H, int32_t d) {
    auto al = [](size_t x) { return (x + 255) / 256 * 256; };
    const int32_t ntiles = (N + 31) / 32;
    const size_t ctiles = (size_t)key_order_ctiles(ntiles);
    int32_t levels, width;
    tree_shape(N, levels, width);
    return 2 * al((size_t)H * N * sizeof(int32_t)) + 2 * al((size_t)H * N * d * sizeof(uint16_t)) +
           al((size_t)H * N * sizeof(uint16_t)) +
           al((size_t)H * width * (2 * d + 2) * sizeof(float)) +
           al((size_t)H * width * kNodeInts * sizeof(int32_t)) + al((size_t)2 * H * sizeof(int32_t)) +
           al((size_t)H * ctiles * (d / 16 + 1) * 64 * 16) +
           al((size_t)H * key_order_wctiles(ctiles) * (d / 16 + 1) * 64 * 16);
}

hipError_t launch_key_order(const void* K, int32_t N, int32_t H, int32_t d, int32_t ntiles, void* ws,
                            KeyOrder* out, hipStream_t stream) {
    auto al = [](size_t x) { return (x + 255) / 256 * 256; };
    const int32_t ctiles = key_order_ctiles(ntiles);
    int32_t levels, width;
    tree_shape(N, levels, width);
    char* p = reinterpret_cast<char*>(ws);
    int32_t* perm_a = reinterpret_cast<int32_t*>(p);
    p += al((size_t)H * N * sizeof(int32_t));
    int32_t* perm_b = reinterpret_cast<int32_t*>(p);
    p += al((size_t)H * N * sizeof(int32_t));
    uint16_t* kp_a = reinterpret_cast<uint16_t*>(p);   // head-major key rows in the current order
    p += al((size_t)H * N * d * sizeof(uint16_t));
    uint16_t* kp_b = reinterpret_cast<uint16_t*>(p);
    p += al((size_t)H * N * d * sizeof(uint16_t));
    uint16_t* code = reinterpret_cast<uint16_t*>(p);
    p += al((size_t)H * N * sizeof(uint16_t));
    float* nodef = reinterpret_cast<float*>(p);
    p += al((size_t)H * width * (2 * d + 2) * sizeof(float));
    int32_t* nodeh = reinterpret_cast<int32_t*>(p);
    p += al((size_t)H * width * kNodeInts * sizeof(int32_t));
    int32_t* votes = reinterpret_cast<int32_t*>(p);
    p += al((size_t)2 * H * sizeof(int32_t));
    uint16_t* bounds = reinterpret_cast<uint16_t*>(p);
    p += al((size_t)H * ctiles * (d / 16 + 1) * 64 * 16);
    uint16_t* wbounds = reinterpret_cast<uint16_t*>(p);
    const int32_t wctiles = key_order_wctiles(ctiles);

    const uint16_t* k = reinterpret_cast<const uint16_t*>(K);
    hipError_t e = launch_fill_zero(reinterpret_cast<float*>(votes), (size_t)2 * H, stream);
    if (e != hipSuccess) return e;
    const dim3 grid((unsigned)((N + 255) / 256), (unsigned)H);
    const dim3 pgrid((unsigned)((N + kBlockPos - 1) / kBlockPos), (unsigned)H);
    if (d == 16)
        hipLaunchKernelGGL(tree_init_kernel<16>, grid, dim3(256), 0, stream, k, N, H, perm_a, kp_a);
    else if (d == 32)
        hipLaunchKernelGGL(tree_init_kernel<32>, grid, dim3(256), 0, stream, k, N, H, perm_a, kp_a);
    else
        hipLaunchKernelGGL(tree_init_kernel<64>, grid, dim3(256), 0, stream, k, N, H, perm_a, kp_a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    int32_t* cur = perm_a;
    int32_t* nxt = perm_b;
    uint16_t* kcur = kp_a;
    uint16_t* knxt = kp_b;
    const int32_t lev0 =
        tree_local_level(N, levels, d == 16 ? kLocalRows<16> : (d == 32 ? kLocalRows<32> : kLocalRows<64>));
    for (int lev = 0; lev < lev0; ++lev) {
        const dim3 ngrid((unsigned)(1 << lev), (unsigned)H);
#define KMIP_TREE_LEVEL(DD)                                                                          \
    hipLaunchKernelGGL(tree_axis_kernel<DD>, ngrid, dim3(64), 0, stream, kcur, N, H, lev, width,     \
                       nodef, nodeh);                                                                \
    if ((e = hipGetLastError()) != hipSuccess) return e;                                             \
    hipLaunchKernelGGL(tree_project_kernel<DD>, pgrid, dim3(256), 0, stream, kcur, N, H, lev, width,   \
                       nodef, nodeh, code);
        if (d == 16) {
            KMIP_TREE_LEVEL(16)
        } else if (d == 32) {
            KMIP_TREE_LEVEL(32)
        } else {
            KMIP_TREE_LEVEL(64)
        }
#undef KMIP_TREE_LEVEL
        if ((e = hipGetLastError()) != hipSuccess) return e;
        hipLaunchKernelGGL(tree_find_kernel, ngrid, dim3(256), 0, stream, N, lev, width, 0, nodeh);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        hipLaunchKernelGGL(tree_hist2_kernel, pgrid, dim3(256), 0, stream, N, lev, width, nodeh, code);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        hipLaunchKernelGGL(tree_find_kernel, ngrid, dim3(256), 0, stream, N, lev, width, 1, nodeh);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if (d == 16)
            hipLaunchKernelGGL(tree_scatter_kernel<16>, pgrid, dim3(256), 0, stream, N, lev, width, nodeh, code,
                               cur, nxt, kcur, knxt);
        else if (d == 32)
            hipLaunchKernelGGL(tree_scatter_kernel<32>, pgrid, dim3(256), 0, stream, N, lev, width, nodeh, code,
                               cur, nxt, kcur, knxt);
        else
            hipLaunchKernelGGL(tree_scatter_kernel<64>, pgrid, dim3(256), 0, stream, N, lev, width, nodeh, code,
                               cur, nxt, kcur, knxt);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        std::swap(cur, nxt);
        std::swap(kcur, knxt);
    }
    if (lev0 < levels) {
        const dim3 lgrid((unsigned)(1 << lev0), (unsigned)H);
        if (d == 16)
            hipLaunchKernelGGL(tree_local_kernel<16>, lgrid, dim3(512), 0, stream, N, lev0, kcur, cur);
        else if (d == 32)
            hipLaunchKernelGGL(tree_local_kernel<32>, lgrid, dim3(512), 0, stream, N, lev0, kcur, cur);
        else
            hipLaunchKernelGGL(tree_local_kernel<64>, lgrid, dim3(512), 0, stream, N, lev0, kcur, cur);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    out->perm = cur;
    out->rows = kcur;
    out->bounds = reinterpret_cast<const uint4*>(bounds);
    out->votes = votes;
    out->ctiles = ctiles;
    out->wbounds = reinterpret_cast<const uint4*>(wbounds);
    out->wctiles = wctiles;
    const dim3 sgrid((unsigned)(ctiles * 32), (unsigned)H);
    const dim3 wgrid((unsigned)(wctiles * 32), (unsigned)H);
    if (d == 16) {
        hipLaunchKernelGGL(sb_bounds_kernel<16>, sgrid, dim3(256), 0, stream, kcur, N, H, ctiles, bounds);
        hipLaunchKernelGGL(win_bounds_kernel<16>, wgrid, dim3(256), 0, stream, kcur, N, H, wctiles, wbounds);
    } else if (d == 32) {
        hipLaunchKernelGGL(sb_bounds_kernel<32>, sgrid, dim3(256), 0, stream, kcur, N, H, ctiles, bounds);
        hipLaunchKernelGGL(win_bounds_kernel<32>, wgrid, dim3(256), 0, stream, kcur, N, H, wctiles, wbounds);
    } else {
        hipLaunchKernelGGL(sb_bounds_kernel<64>, sgrid, dim3(256), 0, stream, kcur, N, H, ctiles, bounds);
        hipLaunchKernelGGL(win_bounds_kernel<64>, wgrid, dim3(256), 0, stream, kcur, N, H, wctiles, wbounds);
    }
    return hipGetLastError();
}

}  // namespace kmip
