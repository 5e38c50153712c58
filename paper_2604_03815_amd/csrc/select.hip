// Fused score + select for k-MIP attention on gfx950 (CDNA4).
//
// Computes, for every query i and head h, the k keys j of i's graph with the
// largest s_ij = q_i . k_j (ties to the lower j): SymbolicMultiply followed by
// RowwiseTopK in Algorithm 1 (Appendix E) of arXiv 2604.03815.  As with the
// symbolic matrices of Appendix F, scores exist only in registers: the kernel
// streams key tiles, forms 32x32 score tiles with one bf16 MFMA per 16 dims
// (fp32 accumulation) and keeps a running top-k per query in LDS.
//
// Work decomposition: an item is QB blocks of 32 query positions of one graph
// and one head; its wave streams every 32-key tile that overlaps the graph.
// Positions map to queries through an optional per-head permutation that
// puts queries of similar direction side by side (group.hip).  One
// wave per workgroup; workgroups are persistent and loop over items.  MFMA operand roles: A = 32 keys x 16 dims, B = 16 dims x 32
// queries, so lane l ends up holding 16 scores of query (l % 32) against keys
//   row(r, l) = 8 * (r / 4) + 4 * (l / 32) + (r % 4),  r = 0..15
// of the tile.  Lanes l and l + 32 share a query.
//
// Selection per query: a loser tree (tournament) over the k best 64-bit
// keys (score code, ~index) in LDS, whose winner is the k-th best; its score
// gives a threshold theta kept in a register.
// Per tile and block each lane reduces its 16 scores with a max3 tree and
// compares once with theta.  Only when some lane's maximum beats theta does
// the wave pick out the scores above theta, append them (with their key
// index) to a per-lane candidate buffer in LDS, and fold the buffers into the
// trees (refreshing theta) whenever one fills up.
//
// Exactness of the filter: theta is the largest float below the k-th best
// score in the tree, so s > theta holds exactly for s >= that score; every
// key that could displace a tree entry, ties included, reaches the rare
// path, and the tree compares full keys (score, then lower index).  The
// result therefore does not depend on the order keys are streamed in, and
// the scan may visit a graph's tiles in any order (used to keep the waves of
// an XCD on the same tiles, see the pacer below).  Keys of
// a tile that lie outside the query's graph are not masked in the streaming
// loop; they can only send a tile down the rare path, which drops them by
// index.
#include <algorithm>
#include <cfloat>

#include "kmip_device.h"
#include "kmip_internal.h"

namespace kmip {
namespace {

__device__ __forceinline__ int tile_row(int r, int half) {
    return 8 * (r >> 2) + 4 * half + (r & 3);
}

// Key tiles are streamed with loads issued from inline assembly, in a fixed
// order, and waited for with explicit vmcnt counts: the compiler may reorder
// ordinary loads of the prefetch ring, and its wait analysis then falls back
// to draining every load before each tile.  vmcnt(n) waits until at most n
// vector-memory operations are outstanding; loads complete in issue order,
// so with n = the number of ring loads issued after the one needed, that load
// has arrived (any other outstanding operation only makes the wait longer).
// The tile address lives in SGPRs, the lane offset in a VGPR.
// The compiler believes an asm load writes its registers at once, so a
// ring register must stay live (be an operand of a later wait) until its
// load has landed; the stream's final drain lists every ring register.
typedef int i32x4 __attribute__((ext_vector_type(4)));

template <int OFF>
__device__ __forceinline__ i32x4 ring_load(const void* tile_base, uint32_t lane_off) {
    i32x4 v;
    asm volatile("global_load_dwordx4 %0, %1, %2 offset:%3"
                 : "=v"(v)
                 : "v"(lane_off), "s"(tile_base), "n"(OFF));
    return v;
}

template <int N>
__device__ __forceinline__ void ring_wait(i32x4& v) {
    asm volatile("s_waitcnt vmcnt(%1)" : "+v"(v) : "n"(N));
}

// acc[r] for a lane-varying r in 0..15, without indexed register access: a
// 4-level tree of bitwise selects (one v_bfi per node) keyed on the bits of
// r.  Written with masks rather than conditionals so that the compiler does
// not turn the tree back into a dynamic vector index.
__device__ __forceinline__ uint32_t bit_mask(int r, int bit) {
    return 0u - (((uint32_t)r >> bit) & 1u);
}

__device__ __forceinline__ uint32_t bsel(uint32_t m, uint32_t x, uint32_t y) {
    return (x & m) | (y & ~m);
}

__device__ __forceinline__ float pick16(const f32x16& a, int r) {
    const uint32_t m3 = bit_mask(r, 3), m2 = bit_mask(r, 2), m1 = bit_mask(r, 1), m0 = bit_mask(r, 0);
    uint32_t v8[8], v4[4], v2[2];
#pragma unroll
    for (int i = 0; i < 8; ++i) v8[i] = bsel(m3, __float_as_uint(a[i + 8]), __float_as_uint(a[i]));
#pragma unroll
    for (int i = 0; i < 4; ++i) v4[i] = bsel(m2, v8[i + 4], v8[i]);
#pragma unroll
    for (int i = 0; i < 2; ++i) v2[i] = bsel(m1, v4[i + 2], v4[i]);
    return __uint_as_float(bsel(m0, v2[1], v2[0]));
}

// Superblock rows of a bound tile whose bound beats a threshold: lane l
// holds m, with bit 15 - r set when its row tile_row(r, l / 32) is needed
// by its query.  ORs m over each half-wave (a prefix OR along each row of
// 16 lanes with DPP shifts, then the rows' last lanes) and returns the
// 32-bit row mask of the tile.
__device__ __forceinline__ uint32_t half_or_rows(uint32_t m) {
    m |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)m, 0x111, 0xF, 0xF, true);   // row_shr:1
    m |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)m, 0x112, 0xF, 0xF, true);   // row_shr:2
    m |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)m, 0x114, 0xF, 0xF, true);   // row_shr:4
    m |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)m, 0x118, 0xF, 0xF, true);   // row_shr:8
    const uint32_t h0 = (uint32_t)__builtin_amdgcn_readlane((int)m, 15) | (uint32_t)__builtin_amdgcn_readlane((int)m, 31);
    const uint32_t h1 = (uint32_t)__builtin_amdgcn_readlane((int)m, 47) | (uint32_t)__builtin_amdgcn_readlane((int)m, 63);
    // bit 15 - r -> bit r, then nibble a (rows 4a .. 4a+3 of the half) to
    // rows 8a .. 8a+3 (half 0) or 8a+4 .. 8a+7 (half 1)
    auto spread = [](uint32_t x) {
        x = __builtin_bitreverse32(x) >> 16;
        return (x & 0xFu) | ((x & 0xF0u) << 4) | ((x & 0xF00u) << 8) | ((x & 0xF000u) << 12);
    };
    return spread(h0) | (spread(h1) << 4);
}

// Loser tree in LDS: column `col` of a [KP][32] array of keys, KP = k rounded
// up to a power of two, 2^lb.  Leaves 0 .. KP-1 (not stored) hold the k best
// keys so far, or sentinels; internal node i (rows 1 .. KP-1) has children
// 2i and 2i+1, leaf L being node KP + L, and stores the loser (the larger
// key) of the match between its children's winners; row 0 holds the overall
// winner, the smallest key.  Replacing the winner by a larger key only
// replays the matches on the winner's path to the root, whose nodes are
// known up front: their loads go out together, one LDS round trip per
// insertion (a 4-ary heap needs one per level).
//
// Tree keys carry their leaf in the low lb bits: the low word ~j of a key
// is shifted up by lb, which drops only one-bits (the sizes accepted keep
// j < 2^31 / max(d, k), so ~j starts with at least lb ones) and keeps the
// order of keys of different j.  A sentinel is leaf L's key L (score word
// 0, below every real key), and a leaf past k - 1 holds kHeapTop, above
// every key, so it never wins.
constexpr uint64_t kHeapTop = ~0ull;

// A selection key in tree form at leaf bits 0.
__device__ __forceinline__ uint64_t tree_key(uint64_t key, int lb) {
    return (key & 0xFFFFFFFF00000000ull) | (uint64_t)((uint32_t)key << lb);
}

// Key index of a tree key; -1 for a sentinel.
__device__ __forceinline__ int32_t tree_index(uint64_t x, int lb) {
    if ((x >> 32) == 0ull) return -1;
    const uint32_t top = lb > 0 ? ~0u << (32 - lb) : 0u;
    return ~(int32_t)(((uint32_t)x >> lb) | top);
}

// Replaces the winner (at leaf `leaf`) by x, which carries that leaf in its
// low bits, and returns the new winner.  The path is LBMAX >= lb levels long
// so that it stays in registers without branches: levels past lb address
// row 0 (node >> i = 0 there), which the caller sets to kHeapTop while it
// keeps the winner in a register, so they never swap.
template <int LBMAX>
__device__ __forceinline__ uint64_t tree_replace(uint64_t* tp, int col, int lb, uint64_t x, int leaf) {
    const int node = (leaf + (1 << lb)) >> 1;
    uint64_t ls[LBMAX];
#pragma unroll
    for (int i = 0; i < LBMAX; ++i) ls[i] = tp[(node >> i) * 32 + col];
#pragma unroll
    for (int i = 0; i < LBMAX; ++i) {
        const bool sw = ls[i] < x;
        const uint64_t lo = sw ? ls[i] : x;
        ls[i] = sw ? x : ls[i];
        x = lo;
    }
#pragma unroll
    for (int i = 0; i < LBMAX; ++i) tp[(node >> i) * 32 + col] = ls[i];
    return x;
}

// The largest float below x, for a finite tree score x; a zero or denormal
// x gives -FLT_MIN instead, so that the threshold is never a denormal (a
// looser threshold only admits a few more candidates).
__device__ __forceinline__ float float_below(float x) {
    const uint32_t b = __float_as_uint(x);
    if ((b & 0x7F800000u) == 0u) return -FLT_MIN;
    return __uint_as_float((int32_t)b >= 0 ? b - 1u : b + 1u);
}

// Pacer of one XCD: a virtual position in a graph's key stream that moves at
// the average speed of that XCD's waves, P(t) = pos + (t - t_ref) * rate
// (tiles per tick of the 100 MHz wall clock).  A wave scans each item's
// tiles chunk by chunk, taking the chunk at P(now) next, so that waves
// which started items at different times still read the same tiles at
// about the same time and share them in the XCD's L2.  Each finished item folds its own speed into rate (moving average)
// and re-anchors (pos, t_ref).  The fields are read and written without
// synchronisation; a torn read only yields a worse start tile, never a
// wrong result.
struct Pacer {
    double pos;
    double rate;
    int64_t t_ref;
    int64_t pad;
};

static_assert(kNumXcd * (sizeof(int32_t) + sizeof(Pacer)) <= kSelectCounterBytes,
              "work counters and pacers must fit their scratch");

// Folds the speed of an item that scanned nt tiles in `ticks` into the pacer.
__device__ __forceinline__ void pacer_update(Pacer* p, int64_t now, int nt, int64_t ticks) {
    if (ticks <= 0) return;
    const double own = (double)nt / (double)ticks;
    const double rate = __hip_atomic_load(&p->rate, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const double pos = __hip_atomic_load(&p->pos, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int64_t t_ref = __hip_atomic_load(&p->t_ref, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    double v = rate > 0.0 ? pos + (double)(now - t_ref) * rate : 0.0;
    if (!(v >= 0.0) || v > 1e15) v = 0.0;
    const double next_rate = rate > 0.0 ? 0.875 * rate + 0.125 * own : own;
    __hip_atomic_store(&p->pos, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&p->t_ref, now, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&p->rate, next_rate, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ uint64_t min_u64(uint64_t a, uint64_t b) { return b < a ? b : a; }

// At least one wave per SIMD: the kernel may use the whole register file
// rather than have the compiler trade registers for occupancy by spilling.
// LBMAX: the loser trees' replay path, at least ceil(log2 k) levels (5 for
// k <= 32, 7 for k <= 128, 8 for k <= 256, 9 for k <= 512); a longer path
// costs the levels it does not need on every insertion.
template <int D, int QB, int SLOTS, int LBMAX>
__global__ __launch_bounds__(64, 1) void select_kernel(
    const uint4* __restrict__ kp, const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
    const Task* __restrict__ tasks, const int32_t* __restrict__ qperm,
    const uint16_t* __restrict__ qlabel, int32_t* __restrict__ seed_ref, const int32_t* __restrict__ kperm,
    const uint4* __restrict__ bounds, const uint4* __restrict__ wbounds, int32_t wctiles,
    int32_t* __restrict__ votes, int32_t ctiles, int32_t ntasks,
    int32_t N, int32_t H, int32_t k, int32_t ntiles, int32_t* __restrict__ work_ctr,
    Pacer* __restrict__ pacers, int32_t* __restrict__ topk_idx) {
    constexpr int NC = D / 16;
    constexpr int TILE_BYTES = NC * 64 * 16;
    constexpr int SBT = kSuperTiles;
    extern __shared__ uint64_t lds[];
    // loser trees of 2^lb leaves, lb <= LBMAX
    static_assert(QB == 1 || LBMAX == 5, "two query blocks take k <= 32");
    const int lb = k <= 1 ? 0 : 32 - __clz(k - 1);
    const int hrows = 1 << lb;
    const uint64_t leaf_mask = (uint64_t)(hrows - 1);

    // Persistent, XCD-aware schedule.  Workgroups are dispatched to the XCDs
    // round-robin; the ones on XCD x take the items of a contiguous range of
    // (head, task) items from that XCD's counter, so an XCD works on one
    // head's keys at a time, and its pacer keeps its waves on the same
    // tiles.  Taking items from a counter balances items of unequal cost and
    // keeps a workgroup that only becomes resident late (when the grid
    // exceeds what fits) from delaying the items it would otherwise own.
    // A wave whose XCD's range is used up goes on with the next XCD's
    // counter, and so on round the XCDs: ranges differ in cost (heads and
    // direction groups prune differently), and without this the XCDs with
    // cheap ranges would sit idle at the end.
    // With grouped queries the counter walks a range with a stride coprime
    // to its length, so that the first items to run cover all direction
    // groups and can seed the items that follow (see below).
    const int items = ntasks * H;
    const int xcd = blockIdx.x % kNumXcd;
    const int items_per_xcd = (items + kNumXcd - 1) / kNumXcd;
    int vx = xcd, visited = 0;
    int item_lo = 0, range = 0, stride = 1;
    auto xcd_range = [&](int x) {
        item_lo = min(items, x * items_per_xcd);
        range = min(items, item_lo + items_per_xcd) - item_lo;
        stride = 1;
        if (qlabel != nullptr && range > 1) {
            stride = max(1, range / max(1, (int)gridDim.x / kNumXcd));
            for (;; ++stride) {
                int a = stride, b = range;
                while (b != 0) {
                    const int r = a % b;
                    a = b;
                    b = r;
                }
                if (a == 1) break;
            }
        }
    };
    xcd_range(vx);
    for (;;) {
    int claim = 0;
    if (threadIdx.x == 0) claim = atomicAdd(&work_ctr[vx], 1);
    claim = __builtin_amdgcn_readfirstlane(claim);
    if (claim >= range) {
        if (++visited == kNumXcd) break;
        vx = vx + 1 == kNumXcd ? 0 : vx + 1;
        xcd_range(vx);
        continue;
    }
    const int item = item_lo + (int)(((int64_t)claim * stride) % range);
    const int head = item / ntasks;
    const int task = item - head * ntasks;

    int q_begin, q_count, key_lo, key_hi;
    if (tasks != nullptr) {
        Task t = tasks[task];
        q_begin = t.q_begin;
        q_count = t.q_count;
        key_lo = t.key_lo;
        key_hi = t.key_hi;
    } else {
        q_begin = task * 32 * QB;
        q_count = min(32 * QB, N - q_begin);
        key_lo = 0;
        key_hi = N;
    }
    // a task without queries (the unused tail of a list filled on the
    // device) has nothing to select
    if (q_count <= 0) continue;

    const int lane = threadIdx.x;
    const int col = lane & 31;
    const int half = lane >> 5;

    uint64_t* trees = lds;                              // [QB][hrows][32] loser trees
    uint64_t* cand = lds + (size_t)QB * hrows * 32;     // [QB][SLOTS][64]

    bf16x8 bq[QB][NC];
    float theta[QB];
    int cnt[QB];
    int32_t qid[QB];
    // |q| rounded up to bf16 (bits), the query's entry of the bound operand
    uint32_t qn_up[QB];
    const int32_t* hperm = qperm != nullptr ? qperm + (size_t)head * N : nullptr;
#pragma unroll
    for (int b = 0; b < QB; ++b) {
        const int qi = 32 * b + col;
        const bool valid = qi < q_count;
        qid[b] = valid ? (hperm != nullptr ? hperm[q_begin + qi] : q_begin + qi) : 0;
        const uint16_t* qrow = Q + ((size_t)qid[b] * H + head) * D + 8 * half;
        float ss = 0.0f;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            uint4 u = valid ? *reinterpret_cast<const uint4*>(qrow + 16 * c) : make_uint4(0, 0, 0, 0);
            bq[b][c] = __builtin_bit_cast(bf16x8, u);
            const uint32_t w4[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float lo = bf16_bits_to_f32(w4[e] & 0xFFFFu), hi = bf16_bits_to_f32(w4[e] >> 16);
                ss = fmaf(lo, lo, ss);
                ss = fmaf(hi, hi, ss);
            }
        }
        ss += __shfl_xor(ss, 32);
        // sqrt in fp32 errs by far less than the 2^-12 added before rounding up
        const uint32_t nb = __float_as_uint(sqrtf(ss) * (1.0f + 0x1p-12f));
        qn_up[b] = (nb >> 16) + ((nb & 0xFFFFu) != 0u ? 1u : 0u);
        theta[b] = valid ? -INFINITY : INFINITY;
        cnt[b] = 0;
    }
    // Empty trees: leaf L holds sentinel L (L < k) or kHeapTop; the winner
    // is leaf 0, and node r keeps the winner of its right subtree, that
    // subtree's leftmost leaf.
    for (int e = lane; e < QB * hrows * 32; e += 64) {
        const int r = (e >> 5) & (hrows - 1);
        uint64_t v = 0ull;
        if (r > 0) {
            const int dep = 31 - __clz(r);
            const int leaf = ((2 * r + 1) << (lb - dep - 1)) - hrows;
            v = leaf < k ? (uint64_t)leaf : kHeapTop;
        }
        trees[e] = v;
    }

    // Seeded thresholds.  Queries of one direction label share most of their
    // top-k keys.  When some query of the label of a block's first query has
    // published its finished top-k row, the block scores its queries against
    // those k keys (one MFMA tile per 32 keys, gathered from K) and starts
    // from theta = the float below each query's lowest such score: k
    // distinct keys of the graph score at least that much, so the query's
    // k-th best does too, and every key that can enter its top-k still
    // passes the filter.  Scores come from the same MFMA on the same
    // operands as in the stream, hence are the same values.  The tree starts
    // empty and fills with keys that pass; theta only ever rises.
    // A block tries the seeds of the labels of its first and of its last
    // query (a block can straddle two labels) and keeps, per query, the
    // larger threshold: each is a valid lower bound of its k-th best.
    if (qlabel != nullptr) {
#pragma unroll
        for (int b = 0; b < QB; ++b) {
            if (32 * b >= q_count) continue;
            const int last = min(31, q_count - 1 - 32 * b);
            int labs[2] = {0, 0};
            if (lane == 0) labs[0] = qlabel[(size_t)head * N + qid[b]];
            if (lane == last) labs[1] = qlabel[(size_t)head * N + qid[b]];
            labs[0] = __builtin_amdgcn_readfirstlane(labs[0]);
            labs[1] = __builtin_amdgcn_readlane(labs[1], last);
            for (int si = 0; si < 2; ++si) {
            if (si == 1 && labs[1] == labs[0]) break;
            int ref = 0;
            if (lane == 0)
                ref = __hip_atomic_load(&seed_ref[(size_t)head * kGroupCenters + labs[si]], __ATOMIC_ACQUIRE,
                                        __HIP_MEMORY_SCOPE_AGENT);
            ref = __builtin_amdgcn_readfirstlane(ref);
            if (ref <= 0 || ref > N) continue;
            const int32_t* srow = topk_idx + ((size_t)(ref - 1) * H + head) * k;
            float low = INFINITY;
            bool ok = true;
            for (int s0 = 0; s0 < k; s0 += 32) {
                const int j = srow[s0 + col < k ? s0 + col : s0];
                ok = ok && j >= 0 && j < N;
                const int jj = (j >= 0 && j < N) ? j : 0;
                const uint4* src = reinterpret_cast<const uint4*>(K + ((size_t)jj * H + head) * D + 8 * half);
                f32x16 sacc = f32x16{};
#pragma unroll
                for (int c = 0; c < NC; ++c)
                    sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        __builtin_bit_cast(bf16x8, src[2 * c]), bq[b][c], sacc, 0, 0, 0);
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    if (s0 + tile_row(r, half) < k) low = fminf(low, sacc[r]);
            }
            low = fminf(low, __shfl_xor(low, 32));
            if (__builtin_amdgcn_ballot_w64(!ok) != 0ull) continue;
            if (theta[b] != INFINITY) theta[b] = fmaxf(theta[b], float_below(low));
            }
        }
    }

    // Fold every lane's candidates into the trees and refresh theta.  With
    // two blocks, each phase has the lower half-wave on one block's trees and
    // the upper half-wave on the other's, so all lanes work on disjoint trees.
    const int32_t* kperm_h = kperm != nullptr ? kperm + (size_t)head * N : nullptr;
    auto merge_all = [&]() {
        if (kperm_h != nullptr) {
            // With a stored key order, candidates carry the key's position in
            // that order; swap in the key's own index before the tree applies
            // its tie rule.  Every slot is looked up (unused ones at position
            // 0) so that all of a lane's loads are in flight together.
            int32_t orig[QB][SLOTS];
#pragma unroll
            for (int b = 0; b < QB; ++b) {
#pragma unroll
                for (int e = 0; e < SLOTS; ++e) {
                    const int pos = e < cnt[b] ? key_index(cand[((size_t)b * SLOTS + e) * 64 + lane]) : 0;
                    orig[b][e] = kperm_h[pos];
                }
            }
#pragma unroll
            for (int b = 0; b < QB; ++b) {
#pragma unroll
                for (int e = 0; e < SLOTS; ++e) {
                    uint64_t* c = &cand[((size_t)b * SLOTS + e) * 64 + lane];
                    if (e < cnt[b]) *c = (*c & 0xFFFFFFFF00000000ull) | (uint32_t)~orig[b][e];
                }
            }
        }
        // (not unrolled: the merge is inlined at every filter site of the
        // unrolled key stream, and one copy of the replay keeps that loop
        // small enough to be unrolled, with its ring registers static)
#pragma unroll 1
        for (int ph = 0; ph < 2; ++ph) {
            const int b = QB == 2 ? (half ^ ph) : 0;
            if (QB == 2 || half == ph) {
                uint64_t* tp = trees + (size_t)b * hrows * 32;
                const uint64_t* cb = cand + (size_t)b * SLOTS * 64;
                const int n = b == 0 ? cnt[0] : cnt[QB - 1];
                // the winner stays in a register; row 0 holds kHeapTop meanwhile
                uint64_t w = tp[col];
                tp[col] = kHeapTop;
                uint64_t c = cb[lane];
                for (int e = 0; e < n; ++e) {
                    // the next candidate's load goes out before this one's replay
                    const uint64_t cn = cb[min(e + 1, SLOTS - 1) * 64 + lane];
                    const uint64_t x = tree_key(c, lb);
                    if (x > w) w = tree_replace<LBMAX>(tp, col, lb, x | (w & leaf_mask), (int)(w & leaf_mask));
                    c = cn;
                }
                tp[col] = w;
            }
            // The trees are private to this wave, whose LDS instructions
            // execute in program order, so the next phase sees this phase's
            // tree writes.  Only compiler reordering has to be fenced off.
            __builtin_amdgcn_wave_barrier();
        }
#pragma unroll
        for (int b = 0; b < QB; ++b) {
            if (theta[b] != INFINITY) {
                const uint64_t root = trees[(size_t)b * hrows * 32 + col];
                theta[b] = fmaxf(theta[b], (root >> 32) == 0ull ? -INFINITY : float_below(key_score(root)));
            }
            cnt[b] = 0;
        }
    };

    // Rare path for block b of the tile starting at key position tbase.
    // Each lane builds a 16-bit mask of its scores above theta, and the wave
    // then walks the set bits: as many rounds as the largest per-lane count,
    // usually one or two.  A lane picks the score of its bit out of its 16
    // registers with a 4-level select on the bits of the register number.  A
    // buffer that fills up is folded between two rounds.
    auto rare_path = [&](const f32x16& acc, int b, int tbase) {
        uint64_t* cb = cand + (size_t)b * SLOTS * 64;
        // Bit 15 - r of mask is set when score r beats theta: theta - s is
        // negative exactly then, and alignbit shifts its sign bit in.
        uint32_t mask = 0;
#pragma unroll
        for (int r = 0; r < 16; ++r)
            mask = __builtin_amdgcn_alignbit(mask, __float_as_uint(theta[b] - acc[r]), 31);
        if (tbase < key_lo || tbase + 32 > key_hi) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int j = tbase + tile_row(r, half);
                if (j < key_lo || j >= key_hi) mask &= ~(1u << (15 - r));
            }
        }
        while (__builtin_amdgcn_ballot_w64(mask != 0u) != 0ull) {
            if (mask != 0u) {
                const int r = 15 - __builtin_ctz(mask);
                mask &= mask - 1u;
                cb[cnt[b] * 64 + lane] = make_key(pick16(acc, r), tbase + tile_row(r, half));
                cnt[b] += 1;
            }
            if (__builtin_amdgcn_ballot_w64(cnt[b] == SLOTS) != 0ull) merge_all();
        }
        __builtin_amdgcn_wave_barrier();
    };

    // ---- Key stream ----
    // The graph's tiles t0 .. t1-1 form nsb superblocks of SBT tiles, and
    // every 64 superblocks form a window.  Superblocks are scanned whole (the
    // last one may run into the next graph's or the padding tiles: such
    // keys only reach the rare path, which drops them by position), window
    // by window, each window's in increasing order, skipping the ones not in
    // the window's mask.
    //
    // Dense mode: every superblock, starting from the one at the XCD's
    // virtual position (single graph) and wrapping around.  Pruned mode
    // (keys stored in superblock order with bounds): a superblock is in the
    // mask when its bound beats the theta of at least one valid query of
    // the wave; theta only rises, so a superblock left out can never hold a
    // key that passes the filter.  Masks of up to 64 windows (a batch) are
    // formed at once, lane w holding window w's.  A head turns to dense
    // mode once seeded items keep finding most superblocks needed (votes).
    const int t0 = key_lo >> 5;
    const int t1 = (key_hi + 31) >> 5;
    const int nt = t1 - t0;
    const int nsb = (nt + SBT - 1) / SBT;
    const int nwin = (nsb + 63) / 64;
    bool pruned = false;
    if (bounds != nullptr) {
        int v = 0;
        if (lane == 0) v = __hip_atomic_load(&votes[head], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        pruned = __builtin_amdgcn_readfirstlane(v) < kDenseVotes;
    }
    const uint4* btiles = bounds != nullptr ? bounds + (size_t)head * ctiles * (NC + 1) * 64 : nullptr;
    const uint4* wtiles = wbounds != nullptr ? wbounds + (size_t)head * wctiles * (NC + 1) * 64 : nullptr;
    uint32_t mask_lo = 0, mask_hi = 0;
    int mask_batch = -1;
    // The last masks compute_batch formed (before a warm-up replaced them):
    // thresholds only rise, so when the same batch is formed again only
    // windows that kept a superblock then can keep one now.
    uint32_t full_lo = 0, full_hi = 0;
    int full_batch = -1;
    // Superblocks of batch 0 already scanned by a warm-up (see below), as
    // window masks held like mask_lo / mask_hi; left out of every mask.
    uint32_t warm_lo = 0, warm_hi = 0;
    // Masks of windows 64 bt .. 64 bt + 63; returns how many superblocks
    // they keep.  With lower, forms no masks and instead raises each query's
    // theta from lower bounds: every key of a superblock also scores at
    // least q.c - |q|_up R (the same MFMA with the sign of |q|_up flipped;
    // the margins that make q.c + |q|_up R an upper bound of the fp32 scores
    // bound the rounding in this direction as well).  A superblock that lies
    // wholly inside the graph holds 256 keys, so when k <= 256 the largest
    // such value over those superblocks is at most the query's k-th best
    // score, and the float below it is a valid theta.  Bound tile g holds superblocks 32 g .. 32 g + 31, scored
    // like key tiles with the query's |q| bound entry as one more chunk; a
    // window's two tiles are loaded while the previous window is scored.
    // With track, each lane also notes, per query block, the superblock of
    // largest bound among its rows (best_sb, -1 for an invalid query).
    int best_sb[QB];
    float best_b[QB];   // with track: each query's largest superblock bound
    auto compute_batch = [&](int bt, bool track, bool lower) {
        const int wlo = bt * 64;
        const int whi = min(nwin, wlo + 64);
        uint64_t mv = 0;
        int needed = 0;
        bf16x8 qa[QB];
        float best_v[QB];
#pragma unroll
        for (int b = 0; b < QB; ++b) {
            qa[b] = __builtin_bit_cast(bf16x8, make_uint4(half == 0 ? (lower ? (qn_up[b] | 0x8000u) : qn_up[b]) : 0u, 0u, 0u, 0u));
            best_v[b] = -INFINITY;
            best_sb[b] = -1;
        }
        uint64_t todo = whi - wlo == 64 ? ~0ull : (1ull << (whi - wlo)) - 1ull;
        if (full_batch == bt && !lower) todo &= __builtin_amdgcn_ballot_w64((full_lo | full_hi) != 0u);
        // Windows whose own bound beats no valid query's theta hold no key
        // that can pass the filter: their bound tiles are not scored (window
        // tile 2 bt + ct holds windows 64 bt + 32 ct .. + 31 as its rows).
        if (wtiles != nullptr && todo != 0ull) {
            bf16x8 qu[QB];
#pragma unroll
            for (int b = 0; b < QB; ++b)
                qu[b] = __builtin_bit_cast(bf16x8, make_uint4(half == 0 ? qn_up[b] : 0u, 0u, 0u, 0u));
            uint64_t wneed = 0;
#pragma unroll
            for (int ct = 0; ct < 2; ++ct) {
                if (((todo >> (32 * ct)) & 0xFFFFFFFFull) == 0ull) continue;
                const uint4* src = wtiles + (size_t)(2 * bt + ct) * (NC + 1) * 64 + lane;
                uint4 wc[NC + 1];
#pragma unroll
                for (int c = 0; c <= NC; ++c) wc[c] = src[c * 64];
                uint32_t lm = 0;
                f32x16 wacc[QB];
#pragma unroll
                for (int b = 0; b < QB; ++b) {
                    wacc[b] = f32x16{};
#pragma unroll
                    for (int c = 0; c < NC; ++c)
                        wacc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, wc[c]), bq[b][c],
                                                                          wacc[b], 0, 0, 0);
                    wacc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, wc[NC]), qu[b],
                                                                      wacc[b], 0, 0, 0);
                }
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    uint32_t any = 0;
#pragma unroll
                    for (int b = 0; b < QB; ++b) any |= __float_as_uint(theta[b] - wacc[b][r]);
                    lm = __builtin_amdgcn_alignbit(lm, any, 31);
                }
                wneed |= (uint64_t)half_or_rows(lm) << (32 * ct);
            }
            todo &= wneed;
        }
        const int nfull = (key_hi - key_lo) / (32 * SBT);
        float low_v[QB];
#pragma unroll
        for (int b = 0; b < QB; ++b) low_v[b] = -INFINITY;
        // Bound tiles of the next windows to score, PD windows ahead (two
        // where registers allow).
        constexpr int PD = NC <= 2 ? 2 : 1;
        uint4 cn[2][NC + 1], cn2[2][NC + 1];
        auto fetch = [&](uint4 (&dst)[2][NC + 1], int w) {
#pragma unroll
            for (int ct = 0; ct < 2; ++ct) {
                const uint4* src = btiles + (size_t)(2 * w + ct) * (NC + 1) * 64 + lane;
#pragma unroll
                for (int c = 0; c <= NC; ++c) dst[ct][c] = src[c * 64];
            }
        };
        if (todo != 0ull) fetch(cn, wlo + (int)__builtin_ctzll(todo));
        if (PD == 2) {
            const uint64_t t1 = todo & (todo - 1ull);
            if (t1 != 0ull) fetch(cn2, wlo + (int)__builtin_ctzll(t1));
        }
        while (todo != 0ull) {
            const int w = wlo + (int)__builtin_ctzll(todo);
            todo &= todo - 1ull;
            uint4 cc[2][NC + 1];
#pragma unroll
            for (int ct = 0; ct < 2; ++ct)
#pragma unroll
                for (int c = 0; c <= NC; ++c) cc[ct][c] = cn[ct][c];
            if (PD == 2) {
#pragma unroll
                for (int ct = 0; ct < 2; ++ct)
#pragma unroll
                    for (int c = 0; c <= NC; ++c) cn[ct][c] = cn2[ct][c];
                const uint64_t t1 = todo & (todo - 1ull);
                if (t1 != 0ull) fetch(cn2, wlo + (int)__builtin_ctzll(t1));
            } else if (todo != 0ull) {
                fetch(cn, wlo + (int)__builtin_ctzll(todo));
            }
            uint64_t m = 0;
#pragma unroll
            for (int ct = 0; ct < 2; ++ct) {
                f32x16 bacc[QB];
#pragma unroll
                for (int b = 0; b < QB; ++b) {
                    bacc[b] = f32x16{};
#pragma unroll
                    for (int c = 0; c < NC; ++c)
                        bacc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, cc[ct][c]),
                                                                          bq[b][c], bacc[b], 0, 0, 0);
                    bacc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, cc[ct][NC]),
                                                                      qa[b], bacc[b], 0, 0, 0);
                }
                if (lower) {
                    const int sb0 = 64 * w + 32 * ct;
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const bool full = sb0 + tile_row(r, half) < nfull;
#pragma unroll
                        for (int b = 0; b < QB; ++b) low_v[b] = full ? fmaxf(low_v[b], bacc[b][r]) : low_v[b];
                    }
                    continue;
                }
                // bit 15 - r: some block's bound beats its theta (theta - bound
                // is negative exactly then; -0 only adds a row)
                uint32_t lm = 0;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    uint32_t any = 0;
#pragma unroll
                    for (int b = 0; b < QB; ++b) any |= __float_as_uint(theta[b] - bacc[b][r]);
                    lm = __builtin_amdgcn_alignbit(lm, any, 31);
                }
                const uint32_t bits = half_or_rows(lm);
                if (track) {
                    // Each query's superblock of largest bound so far (the
                    // first in visiting order among equal ones).  In a tile
                    // of whole superblocks: the largest of the lane's 16
                    // rows by a max3 tree and the first row that holds it;
                    // in the last, row by row, valid rows only.
                    const int sb0 = 64 * w + 32 * ct;
                    if (sb0 + 32 <= nsb) {
#pragma unroll
                        for (int b = 0; b < QB; ++b) {
                            const f32x16& a = bacc[b];
                            const float l0 = fmaxf(fmaxf(a[0], a[1]), a[2]);
                            const float l1 = fmaxf(fmaxf(a[3], a[4]), a[5]);
                            const float l2 = fmaxf(fmaxf(a[6], a[7]), a[8]);
                            const float l3 = fmaxf(fmaxf(a[9], a[10]), a[11]);
                            const float l4 = fmaxf(fmaxf(a[12], a[13]), a[14]);
                            const float mx = fmaxf(fmaxf(fmaxf(l0, l1), l2), fmaxf(fmaxf(l3, l4), a[15]));
                            int pick = 15;
#pragma unroll
                            for (int r = 14; r >= 0; --r) pick = a[r] == mx ? r : pick;
                            const bool better = theta[b] != INFINITY && mx > best_v[b];
                            best_v[b] = better ? mx : best_v[b];
                            best_sb[b] = better ? sb0 + tile_row(pick, half) : best_sb[b];
                        }
                    } else {
#pragma unroll
                        for (int r = 0; r < 16; ++r) {
                            const int sb = sb0 + tile_row(r, half);
#pragma unroll
                            for (int b = 0; b < QB; ++b) {
                                const bool better = sb < nsb && theta[b] != INFINITY && bacc[b][r] > best_v[b];
                                best_v[b] = better ? bacc[b][r] : best_v[b];
                                best_sb[b] = better ? sb : best_sb[b];
                            }
                        }
                    }
                }
                m |= (uint64_t)bits << (32 * ct);
            }
            if (lower) continue;
            const int nv = nsb - 64 * w;
            if (nv < 64) m &= (1ull << nv) - 1ull;
            if (lane == w - wlo) {
                mv = m;
                if (bt == 0) mv &= ~((uint64_t)warm_lo | ((uint64_t)warm_hi << 32));
            }
            needed += __builtin_popcountll(m);
        }
        if (lower) {
#pragma unroll
            for (int b = 0; b < QB; ++b) {
                const float lv = fmaxf(low_v[b], __shfl_xor(low_v[b], 32));
                if (theta[b] != INFINITY && lv > -INFINITY) theta[b] = fmaxf(theta[b], float_below(lv));
            }
            return 0;
        }
        if (track) {
#pragma unroll
            for (int b = 0; b < QB; ++b) best_b[b] = fmaxf(best_v[b], __shfl_xor(best_v[b], 32));
        }
        mask_lo = full_lo = (uint32_t)mv;
        mask_hi = full_hi = (uint32_t)(mv >> 32);
        mask_batch = full_batch = bt;
        return needed;
    };
    auto read_mask = [&](int w) {
        const int l = w - 64 * mask_batch;
        return (uint64_t)(uint32_t)__builtin_amdgcn_readlane(mask_lo, l) |
               ((uint64_t)(uint32_t)__builtin_amdgcn_readlane(mask_hi, l) << 32);
    };
    auto valid_bits = [&](int w) {
        const int nv = nsb - 64 * w;
        return nv >= 64 ? ~0ull : (1ull << nv) - 1ull;
    };

    // Window walk: w is the current window, wm its superblocks not yet
    // taken, wv the number of windows entered after the first.  Dense mode
    // walks a scattered order of the superblocks (virtual superblock v is
    // superblock v * stride_sb mod nsb, stride_sb coprime to nsb), so that
    // the first ones scanned come from all over the stored key order and the
    // thresholds rise early; it starts at virtual superblock s0 and visits
    // window w0 = s0 / 64 once more at the end for its superblocks below s0.
    int w = 0, wv = 0, b0 = 0;
    uint64_t wm = 0;
    int scanned = 0;
    // With unseeded queries, masks are formed again after 16, 64, 256, ...
    // superblocks, as the thresholds rise.
    int stop_at = 0x7FFFFFFF;
    // Warm-up of an item with unseeded queries (one batch of windows): the
    // walk first takes, for every query, the superblock of largest bound,
    // then folds its candidates and forms the masks with the thresholds that
    // gives, leaving out the superblocks already scanned.
    bool warm_pending = false;
    int64_t item_start = 0;
    int stride_sb = 1;
    if (pruned) {
        bool seeded = true;
#pragma unroll
        for (int b = 0; b < QB; ++b) seeded = seeded && __builtin_amdgcn_ballot_w64(theta[b] == -INFINITY) == 0ull;
        // (superblock s holds positions 256 s .. 256 s + 255 when key_lo = 0)
        // With two query blocks (k <= 32), seeded items of a head skip the
        // lower-bound pass once it has raised no threshold in nearly all
        // seeded items of that head (their seeds, k keys of a neighbour's
        // set, are then tighter than the balls' lower bounds): a seeded item
        // whose pass raised nothing votes +1, one whose pass raised a
        // threshold -8, and the pass is skipped from kLowerVotes net votes
        // on.  The votes follow the dense-mode ones, votes[H + head].
        if (key_lo == 0 && k <= 32 * SBT) {
            int lv = 0;
            if (QB == 2 && seeded && lane == 0)
                lv = __hip_atomic_load(&votes[H + head], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (__builtin_amdgcn_readfirstlane(lv) < kLowerVotes) {
                float th0[QB];
#pragma unroll
                for (int b = 0; b < QB; ++b) th0[b] = theta[b];
                compute_batch(0, false, true);
                if (QB == 2 && seeded) {
                    bool raised = false;
#pragma unroll
                    for (int b = 0; b < QB; ++b) raised = raised || __builtin_amdgcn_ballot_w64(theta[b] > th0[b]) != 0ull;
                    if (lane == 0) atomicAdd(&votes[H + head], raised ? -8 : 1);
                }
            }
        }
        const int needed = compute_batch(0, nwin <= 64, false);
        // Seeded items whose masks still keep more than half of the
        // superblocks warm up as well: a poorly seeded query widens the
        // masks of its whole wave.
        const bool warm = nwin <= 64 && (!seeded || 2 * needed > nsb);
        if (warm) {
            // Masks of the union of the best superblocks, one window per lane.
            uint64_t mv = 0;
#pragma unroll
            for (int b = 0; b < QB; ++b) {
                for (;;) {
                    const uint64_t pend = __builtin_amdgcn_ballot_w64(best_sb[b] >= 0);
                    if (pend == 0ull) break;
                    const int sb = __builtin_amdgcn_readlane(best_sb[b], (int)__builtin_ctzll(pend));
                    if (lane == (sb >> 6)) mv |= 1ull << (sb & 63);
#pragma unroll
                    for (int b2 = 0; b2 < QB; ++b2) best_sb[b2] = best_sb[b2] == sb ? -1 : best_sb[b2];
                }
            }
            mask_lo = warm_lo = (uint32_t)mv;
            mask_hi = warm_hi = (uint32_t)(mv >> 32);
            warm_pending = true;
        } else if (!seeded) {
            stop_at = 16;
        } else if (nwin <= 64 && 8 * needed > nsb) {
            // Seeded items whose masks keep more than an eighth of the
            // superblocks warm up on a hot set first: the superblocks whose
            // bound, for some query, lies in the upper half of the gap between
            // that query's theta and its best bound.  The thresholds rise on
            // the likeliest keys, and the masks formed after the warm-up (which
            // leave the hot set out) keep fewer superblocks.
            float th0[QB];
#pragma unroll
            for (int b = 0; b < QB; ++b) {
                th0[b] = theta[b];
                if (theta[b] != INFINITY && best_b[b] > theta[b]) theta[b] = 0.5f * (theta[b] + best_b[b]);
            }
            compute_batch(0, false, false);
#pragma unroll
            for (int b = 0; b < QB; ++b) theta[b] = th0[b];
            full_batch = -1;
            warm_lo = mask_lo;
            warm_hi = mask_hi;
            warm_pending = true;
        }
        if (seeded && lane == 0) atomicAdd(&votes[head], needed * 4 > min(nsb, 64 * 64) * 3 ? 1 : -1);
        wm = read_mask(0);
    } else {
        stride_sb = max(1, (int)((float)nsb * 0.381966f));
        for (;; ++stride_sb) {
            int a = stride_sb, b = nsb;
            while (b != 0) {
                const int r = a % b;
                a = b;
                b = r;
            }
            if (a == 1) break;
        }
        int s0 = 0;
        if (tasks == nullptr) {
            const Pacer* pc = &pacers[xcd];
            const double rate = __hip_atomic_load(&pc->rate, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            const double pos = __hip_atomic_load(&pc->pos, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            const int64_t ref = __hip_atomic_load(&pc->t_ref, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            item_start = wall_clock64();
            const double v = pos + (double)(item_start - ref) * rate;
            if (rate > 0.0 && v >= 0.0 && v < 1e15) s0 = (int)(((int64_t)v / SBT) % nsb);
            s0 = __builtin_amdgcn_readfirstlane(s0);
        }
        w = s0 >> 6;
        b0 = s0 & 63;
        wm = valid_bits(w) & (~0ull << b0);
    }
    const int nvisits = b0 == 0 ? nwin : nwin + 1;
    bool finished = false;

    // Next superblock to scan, into ls.  False when the walk is over
    // (finished) or the masks have to be formed first (a new batch, or
    // stop_at reached); the state is left as is, so a repeated call returns
    // false again until the masks are redone.
    auto next_sb = [&](int& ls) {
        if (scanned >= stop_at) return false;
        while (wm == 0ull) {
            if (wv + 1 >= nvisits) {
                finished = true;
                return false;
            }
            const int wn = w + 1 == nwin ? 0 : w + 1;
            if (pruned && (wn >> 6) != mask_batch) return false;
            ++wv;
            w = wn;
            wm = pruned ? read_mask(w) : valid_bits(w);
            if (wv == nwin) wm &= (1ull << b0) - 1ull;
        }
        ls = 64 * w + (int)__builtin_ctzll(wm);
        if (!pruned) ls = (int)(((int64_t)ls * stride_sb) % nsb);
        wm &= wm - 1ull;
        ++scanned;
        return true;
    };

    const uint32_t lane_off = (uint32_t)lane * 16u;
    const char* head_tiles = reinterpret_cast<const char*>(kp) + (size_t)head * (ntiles + kPadTiles) * TILE_BYTES;
    const char* graph_tiles = head_tiles + (size_t)t0 * TILE_BYTES;

    // Scores of the tile in ring slot `a`; PF - 1 later tiles are in flight
    // (8 chunk loads in all, two whole tiles at d = 128).
    constexpr int PF = NC >= 8 ? 2 : 8 / NC;
    static_assert(SBT % PF == 0, "ring slots must line up with superblocks");
    auto scores = [&](i32x4 (&a)[NC], f32x16 (&acc)[QB]) {
#pragma unroll
        for (int c = 0; c < NC; ++c) ring_wait<(PF - 1) * NC>(a[c]);
#pragma unroll
        for (int b = 0; b < QB; ++b) {
            acc[b] = f32x16{};
#pragma unroll
            for (int c = 0; c < NC; ++c)
                acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    __builtin_bit_cast(bf16x8, a[c]), bq[b][c], acc[b], 0, 0, 0);
        }
    };

    // Largest of a lane's 16 scores: a max3 tree of depth 3 (8 instructions)
    // rather than a chain, so the blocks' reductions interleave.
    auto max16 = [](const f32x16& a) {
        const float l0 = fmaxf(fmaxf(a[0], a[1]), a[2]);
        const float l1 = fmaxf(fmaxf(a[3], a[4]), a[5]);
        const float l2 = fmaxf(fmaxf(a[6], a[7]), a[8]);
        const float l3 = fmaxf(fmaxf(a[9], a[10]), a[11]);
        const float l4 = fmaxf(fmaxf(a[12], a[13]), a[14]);
        return fmaxf(fmaxf(fmaxf(l0, l1), l2), fmaxf(fmaxf(l3, l4), a[15]));
    };

    // Filter the scores of key tile `tile`.
    auto filter = [&](const f32x16 (&acc)[QB], int tile) {
        float m[QB];
#pragma unroll
        for (int b = 0; b < QB; ++b) m[b] = max16(acc[b]);
        uint64_t any = 0;
#pragma unroll
        for (int b = 0; b < QB; ++b) any |= __builtin_amdgcn_ballot_w64(m[b] > theta[b]);
        if (any != 0ull) {
#pragma unroll
            for (int b = 0; b < QB; ++b)
                if (__builtin_amdgcn_ballot_w64(m[b] > theta[b]) != 0ull) rare_path(acc[b], b, tile << 5);
        }
    };

    // Phases: each streams superblocks until next_sb stops, then drains the
    // ring; between phases the masks are formed again.
    for (;;) {
        int ls = 0;
        if (!next_sb(ls)) {
            if (finished && !warm_pending) break;
            // Fold pending candidates so that theta is current, then redo the
            // masks of the batch holding the next window to scan.
            merge_all();
            if (finished) {
                // End of the warm-up: walk every window again with masks
                // that leave out the superblocks it scanned.
                warm_pending = false;
                finished = false;
                stop_at = scanned + 16;
                compute_batch(0, false, false);
                w = 0;
                wv = 0;
                wm = read_mask(0);
                continue;
            }
            if (scanned >= stop_at) stop_at = 4 * scanned;
            const int bt = wm != 0ull ? (w >> 6) : ((w + 1 == nwin ? 0 : w + 1) >> 6);
            compute_batch(bt, false, false);
            if ((w >> 6) == bt) wm &= read_mask(w);
            continue;
        }

        // Prefetch ring: each slot holds one tile, and slot_tile[] remembers
        // which (-1 past the phase's last superblock, whose slots are loaded
        // with the graph's first tile and never filtered).  A slot is
        // refilled with the tile PF positions later as soon as its MFMAs
        // are issued; the load cursor takes the next superblock when it
        // passes the last tile of one (pos is known at each call site).
        bool lex = false;
        i32x4 ring[PF][NC];
        int slot_tile[PF];
        auto refill = [&](i32x4 (&slot)[NC], int& stile, int pos) {
            const int rt = lex ? 0 : ls * SBT + pos;
            stile = lex ? -1 : t0 + rt;
            const char* src = graph_tiles + (size_t)rt * TILE_BYTES;
            slot[0] = ring_load<0>(src, lane_off);
            if constexpr (NC >= 2) slot[1] = ring_load<1024>(src, lane_off);
            if constexpr (NC >= 4) {
                slot[2] = ring_load<2048>(src, lane_off);
                slot[3] = ring_load<3072>(src, lane_off);
            }
            if constexpr (NC >= 8) {
                // (the immediate offset of a global load stays below 4096)
                const char* src2 = src + 4096;
                slot[4] = ring_load<0>(src2, lane_off);
                slot[5] = ring_load<1024>(src2, lane_off);
                slot[6] = ring_load<2048>(src2, lane_off);
                slot[7] = ring_load<3072>(src2, lane_off);
            }
            if (pos == SBT - 1 && !lex) lex = !next_sb(ls);
        };
#pragma unroll
        for (int u = 0; u < PF; ++u) refill(ring[u], slot_tile[u], u);

        // Software pipeline with two accumulator sets: the MFMAs of position
        // p+1 are issued before position p is filtered, so matrix cores and
        // filter overlap.  One pass of the loop body takes one superblock.
        f32x16 acc_a[QB], acc_b[QB];
        int tile_a = slot_tile[0], tile_b = 0;
        scores(ring[0], acc_a);
        refill(ring[0], slot_tile[0], PF % SBT);
        while (tile_a >= 0) {
#pragma unroll
            for (int p = 0; p < SBT; p += 2) {
                const int u1 = (p + 1) % PF, u2 = (p + 2) % PF;
                tile_b = slot_tile[u1];
                scores(ring[u1], acc_b);
                refill(ring[u1], slot_tile[u1], (p + 1 + PF) % SBT);
                filter(acc_a, tile_a);
                tile_a = slot_tile[u2];
                scores(ring[u2], acc_a);
                refill(ring[u2], slot_tile[u2], (p + 2 + PF) % SBT);
                filter(acc_b, tile_b);
            }
        }
        // Drain the ring.  Every ring register is an operand of the wait: a
        // prefetch whose tile is never used is dead to the compiler, which
        // could otherwise hand its registers to other values while the load
        // is still in flight and would land on top of them.
#pragma unroll
        for (int u = 0; u < PF; ++u) {
#pragma unroll
            for (int c = 0; c < NC; ++c) ring_wait<0>(ring[u][c]);
        }
    }
    merge_all();
    if (!pruned && tasks == nullptr && lane == 0) {
        const int64_t now = wall_clock64();
        pacer_update(&pacers[xcd], now, nt, now - item_start);
    }

    // Drain each tree in increasing order into slots k-1 .. 0, which leaves
    // the row sorted by (score desc, index asc); sentinels become -1.  Each
    // winner taken is replaced by kHeapTop, which never wins again.
#pragma unroll
    for (int b = 0; b < QB; ++b) {
        const int qi = 32 * b + col;
        if (half == 0 && qi < q_count) {
            uint64_t* tp = trees + (size_t)b * hrows * 32;
            int32_t* dst = topk_idx + ((size_t)qid[b] * H + head) * k;
            uint64_t w = tp[col];
            tp[col] = kHeapTop;
            for (int p = k - 1; p >= 0; --p) {
                dst[p] = tree_index(w, lb);
                if (p > 0) w = tree_replace<LBMAX>(tp, col, lb, kHeapTop, (int)(w & leaf_mask));
            }
        }
    }
    // Publish the row of the item's first query (drained by lane 0 above) as
    // the seed of its label, unless one is published already.
    if (qlabel != nullptr && lane == 0) {
        __threadfence();
        const int lab = qlabel[(size_t)head * N + qid[0]];
        atomicCAS(&seed_ref[(size_t)head * kGroupCenters + lab], 0, qid[0] + 1);
    }
    // The next item reinitialises the trees this wave just drained.
    __builtin_amdgcn_wave_barrier();
    }  // item loop
}

// Tiles t >= ntiles of each head (the kPadTiles padding) are written as zeros.
// Position p of head h holds key perm[h][p] (key p without perm).
// With rows (the key rows already in the stored order, head-major [H][N][d])
// position p of head h is read from there, in sequence.
__global__ __launch_bounds__(256) void pack_k_kernel(const uint16_t* __restrict__ K,
                                                     const int32_t* __restrict__ perm,
                                                     const uint16_t* __restrict__ rows,
                                                     uint4* __restrict__ kp, int32_t N, int32_t H,
                                                     int32_t nchunk, int32_t ntiles) {
    const int32_t ntiles_all = ntiles + kPadTiles;
    const size_t total = (size_t)H * ntiles_all * nchunk * 64;
    const size_t u = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (u >= total) return;
    const int lane = (int)(u & 63);
    size_t r = u >> 6;
    const int c = (int)(r % nchunk);
    r /= nchunk;
    const int t = (int)(r % ntiles_all);
    const int h = (int)(r / ntiles_all);
    const int pos = t * 32 + (lane & 31);
    uint4 v = make_uint4(0, 0, 0, 0);
    if (pos < N) {
        const int d = nchunk * 16;
        if (rows != nullptr) {
            v = *reinterpret_cast<const uint4*>(rows + ((size_t)h * N + pos) * d + 16 * c + 8 * (lane >> 5));
        } else {
            const int key = perm != nullptr ? perm[(size_t)h * N + pos] : pos;
            v = *reinterpret_cast<const uint4*>(K + ((size_t)key * H + h) * d + 16 * c + 8 * (lane >> 5));
        }
    }
    kp[u] = v;
}

template <int D, int QB, int SLOTS, int LBMAX>
hipError_t launch_select_t(const void* kp, const void* Q, const void* K, const Task* tasks,
                           const QueryGroups* groups, const KeyOrder* keys, int32_t ntasks, int32_t N,
                           int32_t H, int32_t k, int32_t ntiles, int32_t* work_ctr, int32_t* topk_idx,
                           hipStream_t stream, hipEvent_t ev_start, hipEvent_t ev_stop) {
    const int64_t items = (int64_t)ntasks * H;
    const size_t lds = select_lds_bytes(k, SelectShape{QB, SLOTS});
    // One resident wave per workgroup slot of the chip, a multiple of the XCD
    // count, never more workgroups than items.
    // The key-tile loads are asynchronous register writes the compiler does
    // not know about: a spill of a prefetch register would save it before its
    // load lands.  Refuse to run a build in which the kernel uses scratch.
    hipFuncAttributes fa;
    const void* fn = reinterpret_cast<const void*>(select_kernel<D, QB, SLOTS, LBMAX>);
    hipError_t e = hipFuncGetAttributes(&fa, fn);
    if (e != hipSuccess) return e;
    if (fa.localSizeBytes != 0) return hipErrorInvalidDeviceFunction;
    // trees of k > 128 keys take more than 64 KB of LDS (up to 132 KB of
    // the 160 KB a gfx950 workgroup may hold)
    if (lds > 65536 && (e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds)) != hipSuccess)
        return e;
    int dev = 0, cus = 0, per_cu = 0;
    e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e == hipSuccess)
        e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, select_kernel<D, QB, SLOTS, LBMAX>, 64, lds);
    if (e != hipSuccess) return e;
    // work_ctr: kNumXcd item counters, then kNumXcd pacers (all fields 0).
    Pacer* pacers = reinterpret_cast<Pacer*>(work_ctr + kNumXcd);
    const size_t words = (kNumXcd * sizeof(int32_t) + kNumXcd * sizeof(Pacer)) / sizeof(float);
    if ((e = launch_fill_zero(reinterpret_cast<float*>(work_ctr), words, stream)) != hipSuccess) return e;
    const int64_t slots = (int64_t)std::max(cus, 1) * std::max(per_cu, 1);
    const int64_t want = std::min<int64_t>(slots, (items + kNumXcd - 1) / kNumXcd * kNumXcd);
    const int64_t grid = std::max<int64_t>(kNumXcd, want / kNumXcd * kNumXcd);
    if (ev_start != nullptr && (e = hipEventRecord(ev_start, stream)) != hipSuccess) return e;
    hipLaunchKernelGGL((select_kernel<D, QB, SLOTS, LBMAX>), dim3((unsigned)grid), dim3(64), lds, stream,
                       reinterpret_cast<const uint4*>(kp), reinterpret_cast<const uint16_t*>(Q),
                       reinterpret_cast<const uint16_t*>(K), tasks, groups ? groups->perm : nullptr,
                       groups ? groups->label : nullptr, groups ? groups->seed_ref : nullptr,
                       keys ? keys->perm : nullptr, keys ? keys->bounds : nullptr,
                       keys ? keys->wbounds : nullptr, keys ? keys->wctiles : 0,
                       keys ? keys->votes : nullptr, keys ? keys->ctiles : 0, ntasks, N, H, k, ntiles,
                       work_ctr, pacers, topk_idx);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (ev_stop != nullptr) return hipEventRecord(ev_stop, stream);
    return hipSuccess;
}

}  // namespace

size_t select_lds_bytes(int32_t k, SelectShape shape) {
    size_t rows = 1;   // loser-tree rows: k rounded up to a power of two
    while (rows < (size_t)k) rows <<= 1;
    return (size_t)shape.qb * (rows * 32 + (size_t)shape.slots * 64) * sizeof(uint64_t);
}

hipError_t launch_pack_k(const void* K, const int32_t* perm, const uint16_t* rows, void* kp, int32_t N, int32_t H, int32_t d,
                         int32_t ntiles, hipStream_t stream) {
    const int nchunk = d / 16;
    const size_t total = (size_t)H * (ntiles + kPadTiles) * nchunk * 64;
    if (total == 0) return hipSuccess;
    const unsigned blocks = (unsigned)((total + 255) / 256);
    hipLaunchKernelGGL(pack_k_kernel, dim3(blocks), dim3(256), 0, stream,
                       reinterpret_cast<const uint16_t*>(K), perm, rows, reinterpret_cast<uint4*>(kp), N, H,
                       nchunk, ntiles);
    return hipGetLastError();
}

hipError_t launch_select(const void* kp, const void* Q, const void* K, const Task* tasks,
                         const QueryGroups* groups, const KeyOrder* keys, int32_t ntasks, int32_t N,
                         int32_t H, int32_t d, int32_t k, int32_t ntiles, SelectShape shape,
                         int32_t* work_ctr, int32_t* topk_idx, hipStream_t stream,
                         hipEvent_t ev_start, hipEvent_t ev_stop) {
    if (ntasks <= 0) return hipSuccess;
    const int lbmax = k <= 32 ? 5 : k <= 128 ? 7 : k <= 256 ? 8 : 9;
#define KMIP_SELECT_CASE(DD, QQ, SS, LL)                                                         \
    if (d == DD && shape.qb == QQ && shape.slots == SS && lbmax == LL)                           \
        return launch_select_t<DD, QQ, SS, LL>(kp, Q, K, tasks, groups, keys, ntasks, N, H, k, ntiles, \
                                           work_ctr, topk_idx, stream, ev_start, ev_stop);
#define KMIP_SELECT_D(DD)         \
    KMIP_SELECT_CASE(DD, 2, 4, 5) \
    KMIP_SELECT_CASE(DD, 1, 8, 5) \
    KMIP_SELECT_CASE(DD, 1, 8, 7) \
    KMIP_SELECT_CASE(DD, 1, 8, 8) \
    KMIP_SELECT_CASE(DD, 1, 8, 9)
    KMIP_SELECT_D(16)
    KMIP_SELECT_D(32)
    KMIP_SELECT_D(64)
    // d = 128: one query block, k <= 128
    KMIP_SELECT_CASE(128, 1, 8, 5)
    KMIP_SELECT_CASE(128, 1, 8, 7)
#undef KMIP_SELECT_D
#undef KMIP_SELECT_CASE
    return hipErrorInvalidValue;
}

}  // namespace kmip
