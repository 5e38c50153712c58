// Fused score + select for k-MIP attention on gfx950 (CDNA4).
//
// Computes, for every query i and head h, the k keys j of i's graph with the
// largest s_ij = q_i . k_j (ties to the lower j): SymbolicMultiply followed by
// RowwiseTopK in Algorithm 1 (Appendix E) of arXiv 2604.03815.  As with the
// symbolic matrices of Appendix F, scores exist only in registers: the kernel
// streams key tiles, forms 32x32 score tiles with one bf16 MFMA per 16 dims
// (fp32 accumulation) and keeps a running top-k per query in LDS.
//
// Work decomposition: one wave per workgroup handles QB blocks of 32 queries
// of one graph and one head, and streams all 32-key tiles of that graph.
// MFMA operand roles: A = 32 keys x 16 dims, B = 16 dims x 32 queries, so
// lane l ends up holding 16 scores of query (l % 32) against keys
//   row(r, l) = 8 * (r / 4) + 4 * (l / 32) + (r % 4),  r = 0..15
// of the tile.  Lanes l and l + 32 share a query.
//
// Selection per query: a min-heap of the k best 64-bit keys (score code,
// ~index) in LDS whose root gives a threshold theta.  Each lane reduces its
// 16 scores with max3 and compares once with theta; only when some lane
// beats theta does the wave look at individual scores and append the
// winners to a per-lane candidate buffer in LDS.  When a buffer may overflow
// on the next tile, the wave folds the buffers into the heaps (first the
// lanes of the lower half-wave, then the upper one, since they share heaps)
// and refreshes theta.  Keys are streamed in increasing index order, so a
// key whose score equals theta loses the tie to the heap entries and a
// strict comparison is exact; the heap itself orders by the full key.
#include "kmip_device.h"
#include "kmip_internal.h"

namespace kmip {
namespace {

__device__ __forceinline__ int tile_row(int r, int half) {
    return 8 * (r >> 2) + 4 * half + (r & 3);
}

// Min-heap in LDS, column `col` of a [size][32] array of keys.  Places x at
// the root and sifts it down.
__device__ __forceinline__ void heap_sift_down(uint64_t* hp, int col, int size, uint64_t x) {
    int pos = 0;
    for (;;) {
        int l = 2 * pos + 1;
        if (l >= size) break;
        uint64_t cm = hp[l * 32 + col];
        int m = l;
        if (l + 1 < size) {
            uint64_t cr = hp[(l + 1) * 32 + col];
            if (cr < cm) {
                cm = cr;
                m = l + 1;
            }
        }
        if (x <= cm) break;
        hp[pos * 32 + col] = cm;
        pos = m;
    }
    hp[pos * 32 + col] = x;
}

template <int D, int QB>
__global__ __launch_bounds__(64) void select_kernel(
    const uint4* __restrict__ kp, const uint16_t* __restrict__ Q, const Task* __restrict__ tasks,
    int32_t ntasks, int32_t N, int32_t H, int32_t k, int32_t ntiles,
    int32_t* __restrict__ topk_idx) {
    constexpr int NC = D / 16;
    extern __shared__ uint64_t lds[];

    // XCD-aware order: the workgroups that land on one XCD take a contiguous
    // range of (head, task) items, so each XCD's L2 streams few heads.
    const int per_xcd = gridDim.x / kNumXcd;
    const int vid = (blockIdx.x % kNumXcd) * per_xcd + blockIdx.x / kNumXcd;
    if (vid >= ntasks * H) return;
    const int head = vid / ntasks;
    const int task = vid - head * ntasks;

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

    const int lane = threadIdx.x;
    const int col = lane & 31;
    const int half = lane >> 5;

    uint64_t* heaps = lds;                       // [QB][k][32]
    uint64_t* cand = lds + (size_t)QB * k * 32;  // [QB][kCandSlots][64]

    bf16x8 bq[QB][NC];
    float theta[QB];
    int cnt[QB];
#pragma unroll
    for (int b = 0; b < QB; ++b) {
        const int qi = 32 * b + col;
        const bool valid = qi < q_count;
        const uint16_t* qrow = Q + ((size_t)(q_begin + qi) * H + head) * D + 8 * half;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            uint4 u = valid ? *reinterpret_cast<const uint4*>(qrow + 16 * c) : make_uint4(0, 0, 0, 0);
            bq[b][c] = __builtin_bit_cast(bf16x8, u);
        }
        theta[b] = valid ? -INFINITY : INFINITY;
        cnt[b] = 0;
    }
    for (int e = lane; e < QB * k * 32; e += 64) heaps[e] = 0ull;
    __syncthreads();

    auto merge = [&](int b) {
        uint64_t* hp = heaps + (size_t)b * k * 32;
        const uint64_t* cb = cand + (size_t)b * kCandSlots * 64;
#pragma unroll
        for (int ph = 0; ph < 2; ++ph) {
            if (half == ph) {
                const int n = cnt[b];
                for (int e = 0; e < n; ++e) {
                    uint64_t c = cb[e * 64 + lane];
                    if (c > hp[col]) heap_sift_down(hp, col, k, c);
                }
            }
            __syncthreads();
        }
        if (theta[b] != INFINITY) {
            uint64_t root = hp[col];
            theta[b] = root == 0ull ? -INFINITY : key_score(root);
        }
        cnt[b] = 0;
    };

    const int t0 = key_lo >> 5;
    const int t1 = (key_hi + 31) >> 5;
    const uint4* kbase = kp + (size_t)head * ntiles * NC * 64 + lane;

    // Prefetch ring of key tiles in registers; loads past the last tile are
    // clamped to it (harmless repeats, never out of bounds).
    constexpr int PF = 8 / NC;
    uint4 ring[PF][NC];
#pragma unroll
    for (int u = 0; u < PF; ++u) {
        const int tt = min(t0 + u, t1 - 1);
#pragma unroll
        for (int c = 0; c < NC; ++c) ring[u][c] = kbase[((size_t)tt * NC + c) * 64];
    }

    auto scores = [&](const uint4 (&a)[NC], f32x16 (&acc)[QB]) {
#pragma unroll
        for (int b = 0; b < QB; ++b) {
            acc[b] = f32x16{};
#pragma unroll
            for (int c = 0; c < NC; ++c)
                acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    __builtin_bit_cast(bf16x8, a[c]), bq[b][c], acc[b], 0, 0, 0);
        }
    };

    auto filter = [&](f32x16 (&acc)[QB], int t) {
        const int tbase = t << 5;
        if (tbase < key_lo || tbase + 32 > key_hi) {
            // Tile straddles the graph boundary: keys outside never qualify.
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int j = tbase + tile_row(r, half);
                if (j < key_lo || j >= key_hi) {
#pragma unroll
                    for (int b = 0; b < QB; ++b) acc[b][r] = -INFINITY;
                }
            }
        }
#pragma unroll
        for (int b = 0; b < QB; ++b) {
            float m = fmaxf(fmaxf(acc[b][0], acc[b][1]), acc[b][2]);
#pragma unroll
            for (int r = 3; r < 15; r += 2) m = fmaxf(fmaxf(m, acc[b][r]), acc[b][r + 1]);
            m = fmaxf(m, acc[b][15]);
            if (__builtin_amdgcn_ballot_w64(m > theta[b]) != 0ull) {
                uint64_t* cb = cand + (size_t)b * kCandSlots * 64;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const bool hit = acc[b][r] > theta[b];
                    if (__builtin_amdgcn_ballot_w64(hit) != 0ull) {
                        if (hit) {
                            cb[cnt[b] * 64 + lane] = make_key(acc[b][r], tbase + tile_row(r, half));
                            cnt[b] += 1;
                        }
                    }
                }
                if (__builtin_amdgcn_ballot_w64(cnt[b] > kCandSlots - 16) != 0ull) merge(b);
            }
        }
    };

    // Software pipeline: the MFMAs of tile t+1 are issued before tile t is
    // filtered, so the matrix cores and the filter overlap.
    f32x16 acc_next[QB];
    scores(ring[0], acc_next);
    {
        const int tt = min(t0 + PF, t1 - 1);
#pragma unroll
        for (int c = 0; c < NC; ++c) ring[0][c] = kbase[((size_t)tt * NC + c) * 64];
    }
    for (int t = t0; t < t1; t += PF) {
#pragma unroll
        for (int u = 0; u < PF; ++u) {
            const int tc = t + u;
            if (tc >= t1) break;
            f32x16 acc[QB];
#pragma unroll
            for (int b = 0; b < QB; ++b) acc[b] = acc_next[b];
            const int un = (u + 1) % PF;
            if (tc + 1 < t1) {
                scores(ring[un], acc_next);
                const int tt = min(tc + 1 + PF, t1 - 1);
#pragma unroll
                for (int c = 0; c < NC; ++c) ring[un][c] = kbase[((size_t)tt * NC + c) * 64];
            }
            filter(acc, tc);
        }
    }

#pragma unroll
    for (int b = 0; b < QB; ++b) {
        if (__builtin_amdgcn_ballot_w64(cnt[b] > 0) != 0ull) merge(b);
    }

    // Drain each heap in increasing order into slots k-1 .. 0, which leaves
    // the row sorted by (score desc, index asc); sentinels become -1.
#pragma unroll
    for (int b = 0; b < QB; ++b) {
        const int qi = 32 * b + col;
        if (half == 0 && qi < q_count) {
            uint64_t* hp = heaps + (size_t)b * k * 32;
            int32_t* dst = topk_idx + ((size_t)(q_begin + qi) * H + head) * k;
            for (int p = k - 1; p >= 0; --p) {
                dst[p] = key_index(hp[col]);
                if (p > 0) heap_sift_down(hp, col, p, hp[p * 32 + col]);
            }
        }
    }
}

__global__ __launch_bounds__(256) void pack_k_kernel(const uint16_t* __restrict__ K,
                                                     uint4* __restrict__ kp, int32_t N, int32_t H,
                                                     int32_t nchunk, int32_t ntiles) {
    const size_t total = (size_t)H * ntiles * nchunk * 64;
    const size_t u = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (u >= total) return;
    const int lane = (int)(u & 63);
    size_t r = u >> 6;
    const int c = (int)(r % nchunk);
    r /= nchunk;
    const int t = (int)(r % ntiles);
    const int h = (int)(r / ntiles);
    const int key = t * 32 + (lane & 31);
    uint4 v = make_uint4(0, 0, 0, 0);
    if (key < N) {
        const int d = nchunk * 16;
        v = *reinterpret_cast<const uint4*>(K + ((size_t)key * H + h) * d + 16 * c + 8 * (lane >> 5));
    }
    kp[u] = v;
}

template <int D, int QB>
hipError_t launch_select_t(const void* kp, const void* Q, const Task* tasks, int32_t ntasks,
                           int32_t N, int32_t H, int32_t k, int32_t ntiles, int32_t* topk_idx,
                           hipStream_t stream) {
    const int64_t items = (int64_t)ntasks * H;
    const int64_t grid = (items + kNumXcd - 1) / kNumXcd * kNumXcd;
    const size_t lds = select_lds_bytes(k, QB);
    hipLaunchKernelGGL((select_kernel<D, QB>), dim3((unsigned)grid), dim3(64), lds, stream,
                       reinterpret_cast<const uint4*>(kp), reinterpret_cast<const uint16_t*>(Q),
                       tasks, ntasks, N, H, k, ntiles, topk_idx);
    return hipGetLastError();
}

}  // namespace

size_t select_lds_bytes(int32_t k, int32_t qb) {
    return (size_t)qb * ((size_t)k * 32 + (size_t)kCandSlots * 64) * sizeof(uint64_t);
}

hipError_t launch_pack_k(const void* K, void* kp, int32_t N, int32_t H, int32_t d, int32_t ntiles,
                         hipStream_t stream) {
    const int nchunk = d / 16;
    const size_t total = (size_t)H * ntiles * nchunk * 64;
    if (total == 0) return hipSuccess;
    const unsigned blocks = (unsigned)((total + 255) / 256);
    hipLaunchKernelGGL(pack_k_kernel, dim3(blocks), dim3(256), 0, stream,
                       reinterpret_cast<const uint16_t*>(K), reinterpret_cast<uint4*>(kp), N, H,
                       nchunk, ntiles);
    return hipGetLastError();
}

hipError_t launch_select(const void* kp, const void* Q, const Task* tasks, int32_t ntasks,
                         int32_t N, int32_t H, int32_t d, int32_t k, int32_t ntiles, int32_t qb,
                         int32_t* topk_idx, hipStream_t stream) {
    if (ntasks <= 0) return hipSuccess;
#define KMIP_SELECT_CASE(DD, QQ)                                                                 \
    if (d == DD && qb == QQ)                                                                     \
        return launch_select_t<DD, QQ>(kp, Q, tasks, ntasks, N, H, k, ntiles, topk_idx, stream);
    KMIP_SELECT_CASE(16, 1)
    KMIP_SELECT_CASE(16, 2)
    KMIP_SELECT_CASE(32, 1)
    KMIP_SELECT_CASE(32, 2)
    KMIP_SELECT_CASE(64, 1)
    KMIP_SELECT_CASE(64, 2)
#undef KMIP_SELECT_CASE
    return hipErrorInvalidValue;
}

}  // namespace kmip
