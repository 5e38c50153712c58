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
//      such prefix with at least k' keys at or above it.  The keys at or
//      above T are the candidates: the k' best and the few others that share
//      the k'-th best's 16-bit prefix;
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
    uint32_t T = 0;
    for (int bit = 31; bit >= 16; --bit)
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
    const int nc = group_sum(mine);
    __syncthreads();   // every score is in registers: the LDS is reused for the candidates

    // 4. the candidates of each query, listed in LDS, then placed by rank
    uint64_t* kept = reinterpret_cast<uint64_t*>(sc);   // [32][kSmallKept] (code, ~index)
    if (active) {
        int slot = q * kSmallKept + pre - mine;
#pragma unroll
        for (int i = 0; i < kSmallPer; ++i)
            if (take(i)) kept[slot++] = ((uint64_t)code[i] << 32) | (uint32_t)(~(s + kSmallTpq * i));
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
    static_assert((size_t)32 * kSmallKept * 8 <= sizeof(float) * kSmallGraph * kSmallStride,
                  "the kept keys fit the score area");
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
