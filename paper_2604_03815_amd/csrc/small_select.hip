// Score + select for the small graphs of a block-diagonal batch on gfx950.
//
// RowwiseTopK of Algorithm 1 (Appendix E) of arXiv 2604.03815 for graphs of
// at most kSmallGraph nodes.  There a query keeps a large share of its graph
// (k / n of several percent), so a running threshold filters little and the
// streaming kernel spends its time inserting into its trees.  Instead, a
// workgroup of 512 threads takes one task (up to 32 queries of one graph and
// one head):
//   1. its eight waves form the scores of the 32 queries against every key
//      of the graph with the streaming kernel's MFMA on the same tiled key
//      operands, so the fp32 scores are the same values, and keep them in LDS
//      ([key][query], row stride 33 words: the stores of a wave and the reads
//      of a query's threads are free of bank conflicts);
//   2. sixteen threads per query hold its scores as order-preserving 32-bit
//      codes (larger score, larger code) and fix the top 16 bits of the code
//      T of the k'-th best key, k' = min(k, n), bit by bit: T is the largest
//      such prefix with at least k' keys at or above it.  The leading bits
//      that the largest code and a lower bound L of the k'-th best share (for
//      k' <= 16 the k'-th largest of the threads' own maxima) are fixed at
//      once, and when at most kSmallList keys reach L with its low 16 bits
//      cleared (every candidate does), the threads list those keys in LDS,
//      seven a thread, and the search and the steps below run on the list.
//      The keys at or above T are the candidates: the k' best and the few
//      others that share the k'-th best's 16-bit prefix;
//   3. when more than kSmallKept keys are candidates (many exact ties), the
//      low 16 bits are fixed as well, giving the k'-th best code exactly, and
//      the candidates are the keys above it plus, at it, the ones of lowest
//      index that the row still needs (the tie rule: score descending, index
//      ascending), found by bisection on the index;
//   4. the candidates are listed per query (prefix sums over its threads), and
//      a candidate's place in the row is the number of candidates that beat
//      it (higher score, or the same score and a lower index); those placed
//      before k' are written, so the row comes out sorted; slots k'..k-1 get
//      -1.
#include "kmip_device.h"
#include "kmip_internal.h"

namespace kmip {
namespace {

constexpr int kSmallStride = 33;                     // LDS words per key row of scores
constexpr int kSmallKept = KMIP_MAX_K_WIDE;          // candidates listed per query (k <= this)
constexpr int kSmallList = 112;                      // keys listed per query above the lower bound
constexpr int kSmallTpq = 16;                        // threads per query
constexpr int kSmallThreads = 32 * kSmallTpq;
constexpr int kSmallPer = (kSmallGraph + kSmallTpq - 1) / kSmallTpq;   // codes per thread

__device__ __forceinline__ int small_tile_row(int r, int half) {
    return 8 * (r >> 2) + 4 * half + (r & 3);
}

// The threads of a query are one row of 16 lanes, so their sums and scans
// use DPP row operations (a VALU modifier) rather than LDS permutes.
static_assert(kSmallTpq == 16, "a query's threads are one DPP row");

// Sum over the 16 threads of a query: quad swaps, then the half-row and row
// mirrors (each pairs lanes of the two halves it joins).
__device__ __forceinline__ int group_sum(int v) {
    v += __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false);    // quad_perm [1,0,3,2]
    v += __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false);    // quad_perm [2,3,0,1]
    v += __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false);   // row_half_mirror
    v += __builtin_amdgcn_update_dpp(0, v, 0x140, 0xF, 0xF, false);   // row_mirror
    return v;
}

// Inclusive prefix sum over the 16 threads of a query (row shifts, zero
// shifted in).
__device__ __forceinline__ int group_scan(int v) {
    v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, true);    // row_shr:1
    v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, true);    // row_shr:2
    v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, true);    // row_shr:4
    v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, true);    // row_shr:8
    return v;
}

// Largest value over the 16 threads of a query, with the same row operations.
__device__ __forceinline__ uint32_t group_max(uint32_t v) {
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false));
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false));
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xF, 0xF, false));
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x140, 0xF, 0xF, false));
    return v;
}

// The kk-th largest of the 16 threads' values v (kk <= 16): the value of the
// threads with fewer than kk values above theirs and at least kk at or
// above (row rotations bring every other thread's value).
__device__ __forceinline__ uint32_t group_kth(uint32_t v, int kk) {
    int gt = 0, ge = 1;
#define KMIP_ROR(R)                                                                       \
    {                                                                                     \
        const uint32_t o = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x120 + R, 0xF, 0xF, false); \
        gt += o > v ? 1 : 0;                                                              \
        ge += o >= v ? 1 : 0;                                                             \
    }
    KMIP_ROR(1) KMIP_ROR(2) KMIP_ROR(3) KMIP_ROR(4) KMIP_ROR(5) KMIP_ROR(6) KMIP_ROR(7) KMIP_ROR(8)
    KMIP_ROR(9) KMIP_ROR(10) KMIP_ROR(11) KMIP_ROR(12) KMIP_ROR(13) KMIP_ROR(14) KMIP_ROR(15)
#undef KMIP_ROR
    return group_max(gt < kk && ge >= kk ? v : 0u);
}

template <int D>
__global__ __launch_bounds__(kSmallThreads) void small_select_kernel(const uint4* __restrict__ kp, const uint16_t* __restrict__ Q,
                                                           const Task* __restrict__ tasks, int32_t ntasks, int32_t N,
                                                           int32_t H, int32_t k, int32_t ntiles,
                                                           int32_t* __restrict__ topk_idx) {
    constexpr int NC = D / 16;
    constexpr int TILE_BYTES = NC * 64 * 16;
    constexpr int kMaxTiles = kSmallGraph / 32 + 1;   // tiles a graph can touch
    constexpr int kWaves = kSmallThreads / 64;
    constexpr int kWaveTiles = (kMaxTiles + kWaves - 1) / kWaves;
    __shared__ float sc[kSmallGraph * kSmallStride];
    const int t = threadIdx.x;
    const int wave = t >> 6, lane = t & 63;
    const int col = lane & 31, half = lane >> 5;
    const int head = blockIdx.x / ntasks;
    const Task tk = tasks[blockIdx.x - head * ntasks];
    const int n = tk.key_hi - tk.key_lo;

    // 1. scores of the task's queries (columns) against the graph's keys
    bf16x8 bq[NC];
    {
        const bool valid = col < tk.q_count;
        const uint16_t* qrow = Q + ((size_t)(valid ? tk.q_begin + col : 0) * H + head) * D + 8 * half;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            const uint4 u = valid ? *reinterpret_cast<const uint4*>(qrow + 16 * c) : make_uint4(0, 0, 0, 0);
            bq[c] = __builtin_bit_cast(bf16x8, u);
        }
    }
    const char* head_tiles = reinterpret_cast<const char*>(kp) + (size_t)head * (ntiles + kPadTiles) * TILE_BYTES;
    const int t0 = tk.key_lo >> 5, nt = ((tk.key_hi + 31) >> 5) - t0;
    uint4 tw[kWaveTiles][NC];   // this wave's tiles, all loads in flight together
#pragma unroll
    for (int u = 0; u < kWaveTiles; ++u) {
        const int tt = wave + kWaves * u;
        if (tt < nt) {
            const uint4* src = reinterpret_cast<const uint4*>(head_tiles + (size_t)(t0 + tt) * TILE_BYTES) + lane;
#pragma unroll
            for (int c = 0; c < NC; ++c) tw[u][c] = src[c * 64];
        }
    }
#pragma unroll
    for (int u = 0; u < kWaveTiles; ++u) {
        const int tt = wave + kWaves * u;
        if (tt < nt) {
            f32x16 acc = f32x16{};
#pragma unroll
            for (int c = 0; c < NC; ++c)
                acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, tw[u][c]), bq[c], acc, 0, 0, 0);
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int j = 32 * (t0 + tt) + small_tile_row(r, half) - tk.key_lo;
                if (j >= 0 && j < n) sc[j * kSmallStride + col] = acc[r];
            }
        }
    }
    __syncthreads();

    // 2. codes of the row, kSmallTpq threads per query, and the top half of T
    const int q = t / kSmallTpq, s = t % kSmallTpq;
    const bool active = q < tk.q_count;
    uint32_t code[kSmallPer];
#pragma unroll
    for (int i = 0; i < kSmallPer; ++i) {
        const int j = s + kSmallTpq * i;
        // 0 lies below every score's code (that of -inf is 0x007FFFFF)
        code[i] = active && j < n ? score_code(sc[j * kSmallStride + q]) : 0u;
    }
    const int kk = n < k ? n : k;
    auto count_at_least = [&](uint32_t x) {
        int c = 0;
#pragma unroll
        for (int i = 0; i < kSmallPer; ++i) c += code[i] >= x ? 1 : 0;
        return group_sum(c);
    };
    // The k'-th best code lies between a lower bound L (for k' <= 16 the
    // k'-th largest of the threads' maxima, which k' keys reach; else 0) and
    // the largest code U, so it shares their common leading bits, and the
    // bit-by-bit search starts below them.
    uint32_t mx = 0;
#pragma unroll
    for (int i = 0; i < kSmallPer; ++i) mx = max(mx, code[i]);
    const uint32_t U = group_max(mx);
    const uint32_t L = kk <= kSmallTpq ? group_kth(mx, kk) : 0u;
    const uint32_t diff = L ^ U;
    const int top = diff == 0u ? -1 : 31 - __clz(diff);
    uint32_t T = top < 0 ? U : top >= 31 ? 0u : U & ~((2u << top) - 1u);
    T &= 0xFFFF0000u;
    // T is the k'-th best code's 16-bit prefix and that code is at least L,
    // so T, and with it every candidate's code, is at least L with its low
    // 16 bits cleared (Lc).  When at most kSmallList keys reach Lc, the
    // query's threads list them (7 a thread) and search and select on the
    // list alone: for any x >= Lc the list holds every code >= x, and below
    // Lc both counts reach k'.
    const uint32_t Lc = L & 0xFFFF0000u;
    int lm = 0;
#pragma unroll
    for (int i = 0; i < kSmallPer; ++i) lm += code[i] >= Lc && code[i] != 0u ? 1 : 0;
    const int lpre = group_scan(lm);
    const bool use_list = group_sum(lm) <= kSmallList;   // the same for a query's threads
    __syncthreads();   // every score is in registers: the LDS is reused

    // 4. the candidates of each query, listed in LDS, then placed by rank
    uint64_t* kept = reinterpret_cast<uint64_t*>(sc);   // [32][kSmallKept] (code, ~index)
    uint64_t* lst = kept + 32 * kSmallKept;             // [32][kSmallList]
    if (use_list) {
        int slot = q * kSmallList + lpre - lm;
#pragma unroll
        for (int i = 0; i < kSmallPer; ++i)
            if (code[i] >= Lc && code[i] != 0u)
                lst[slot++] = ((uint64_t)code[i] << 32) | (uint32_t)(~(s + kSmallTpq * i));
    }
    __syncthreads();
    int nc = 0;
    if (use_list) {
        const int m = group_sum(lm);
        uint64_t e[kSmallList / kSmallTpq];
#pragma unroll
        for (int r = 0; r < kSmallList / kSmallTpq; ++r)
            e[r] = s + kSmallTpq * r < m ? lst[q * kSmallList + s + kSmallTpq * r] : 0ull;
        auto list_at_least = [&](uint32_t x) {
            int c = 0;
#pragma unroll
            for (int r = 0; r < kSmallList / kSmallTpq; ++r) c += (uint32_t)(e[r] >> 32) >= x ? 1 : 0;
            return group_sum(c);
        };
        for (int bit = min(top, 31); bit >= 16; --bit)
            if (list_at_least(T | (1u << bit)) >= kk) T |= 1u << bit;
        // at most kSmallList keys reach T: no exact pass
        int mine = 0;
#pragma unroll
        for (int r = 0; r < kSmallList / kSmallTpq; ++r) mine += (uint32_t)(e[r] >> 32) >= T && e[r] != 0ull ? 1 : 0;
        const int pre = group_scan(mine);
        nc = group_sum(mine);
        if (active) {
            int slot = q * kSmallKept + pre - mine;
#pragma unroll
            for (int r = 0; r < kSmallList / kSmallTpq; ++r)
                if ((uint32_t)(e[r] >> 32) >= T && e[r] != 0ull) kept[slot++] = e[r];
        }
    } else {
        for (int bit = min(top, 31); bit >= 16; --bit)
            if (count_at_least(T | (1u << bit)) >= kk) T |= 1u << bit;
        // 3. many candidates: the exact k'-th best code and the ties at it
        const bool exact = count_at_least(T) > kSmallKept;
        int m = 0;
        if (exact) {
            for (int bit = 15; bit >= 0; --bit)
                if (count_at_least(T | (1u << bit)) >= kk) T |= 1u << bit;
            int above = 0;
#pragma unroll
            for (int i = 0; i < kSmallPer; ++i) above += code[i] > T ? 1 : 0;
            const int need = kk - group_sum(above);
            if (need > 0) {
                // the smallest m such that the keys at T with index below m
                // complete the row
                int lo = 0, hi = n;
                while (hi - lo > 1) {
                    const int mid = (lo + hi) >> 1;
                    int c = 0;
#pragma unroll
                    for (int i = 0; i < kSmallPer; ++i) c += (code[i] == T && s + kSmallTpq * i < mid) ? 1 : 0;
                    if (group_sum(c) >= need) hi = mid; else lo = mid;
                }
                m = hi;
            }
        }
        auto take = [&](int i) {
            const int j = s + kSmallTpq * i;
            return exact ? (code[i] > T || (code[i] == T && code[i] != 0u && j < m)) : (code[i] >= T && code[i] != 0u);
        };
        int mine = 0;
#pragma unroll
        for (int i = 0; i < kSmallPer; ++i) mine += take(i) ? 1 : 0;
        // inclusive prefix sum over the query's threads, and their total
        const int pre = group_scan(mine);
        nc = group_sum(mine);
        if (active) {
            int slot = q * kSmallKept + pre - mine;
#pragma unroll
            for (int i = 0; i < kSmallPer; ++i)
                if (take(i)) kept[slot++] = ((uint64_t)code[i] << 32) | (uint32_t)(~(s + kSmallTpq * i));
        }
    }
    __syncthreads();
    if (active) {
        int32_t* dst = topk_idx + ((size_t)(tk.q_begin + q) * H + head) * k;
        const uint64_t* row = kept + q * kSmallKept;
        for (int e = s; e < nc; e += kSmallTpq) {
            const uint64_t x = row[e];
            int rank = 0;
            for (int f = 0; f < nc; ++f) rank += row[f] > x ? 1 : 0;
            if (rank < kk) dst[rank] = tk.key_lo + key_index(x);
        }
        for (int p = kk + s; p < k; p += kSmallTpq) dst[p] = -1;
    }
}

}  // namespace

hipError_t launch_small_select(const void* kp, const void* Q, const Task* tasks, int32_t ntasks, int32_t N,
                               int32_t H, int32_t d, int32_t k, int32_t ntiles, int32_t* topk_idx,
                               hipStream_t stream) {
    if (ntasks <= 0) return hipSuccess;
    static_assert((size_t)32 * (kSmallKept + kSmallList) * 8 <= sizeof(float) * kSmallGraph * kSmallStride,
                  "the kept keys and the lists fit the score area");
    if (k > kSmallKept) return hipErrorInvalidValue;
    const dim3 grid((unsigned)((int64_t)ntasks * H));
    const uint4* kpp = reinterpret_cast<const uint4*>(kp);
    const uint16_t* q = reinterpret_cast<const uint16_t*>(Q);
    switch (d) {
        case 16:
            hipLaunchKernelGGL(small_select_kernel<16>, grid, dim3(kSmallThreads), 0, stream, kpp, q, tasks, ntasks, N, H, k,
                               ntiles, topk_idx);
            break;
        case 32:
            hipLaunchKernelGGL(small_select_kernel<32>, grid, dim3(kSmallThreads), 0, stream, kpp, q, tasks, ntasks, N, H, k,
                               ntiles, topk_idx);
            break;
        case 64:
            hipLaunchKernelGGL(small_select_kernel<64>, grid, dim3(kSmallThreads), 0, stream, kpp, q, tasks, ntasks, N, H, k,
                               ntiles, topk_idx);
            break;
        default:
            return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace kmip
