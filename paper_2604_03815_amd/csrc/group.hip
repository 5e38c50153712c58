// Query grouping for the score+select kernel.
//
// Which keys win the top-k of a query depends only on the query's direction
// (scaling q by a positive factor scales every score alike).  Queries that
// point the same way therefore share most of their top-k keys, and a wave
// that holds such queries sees its running thresholds rise together and sends
// far fewer key tiles down the selection path.  Per head, every query is
// labelled with the nearest (largest cosine) of kGroupCenters reference
// directions, taken from an evenly strided sample of the queries, and the
// queries are stably bucketed by label.  The result is a permutation of the
// query positions per head; the select kernel reads query perm[h][p] for
// position p and writes that query's own output row, so the results do not
// depend on the grouping at all, only the speed does.
#include "kmip_device.h"
#include "kmip_internal.h"

namespace kmip {
namespace {

constexpr int C = kGroupCenters;

// centers[h][c][:] = unit vector of query row floor((2c+1) N / 2C) of head h
// (zero if that row is zero), rounded to bf16 (nearest even).
__global__ __launch_bounds__(256) void group_centers_kernel(const uint16_t* __restrict__ Q,
                                                            int32_t N, int32_t H, int32_t d,
                                                            uint16_t* __restrict__ centers) {
    const int c = threadIdx.x;
    const int h = blockIdx.x;
    const int64_t row = ((int64_t)(2 * c + 1) * N) / (2 * C);
    const uint16_t* q = Q + ((size_t)row * H + h) * d;
    float ss = 0.0f;
    for (int t = 0; t < d; ++t) {
        const float x = bf16_bits_to_f32(q[t]);
        ss = fmaf(x, x, ss);
    }
    const float inv = ss > 0.0f ? rsqrtf(ss) : 0.0f;
    uint16_t* dst = centers + ((size_t)h * C + c) * d;
    for (int t = 0; t < d; ++t) {
        const uint32_t b = __float_as_uint(bf16_bits_to_f32(q[t]) * inv);
        dst[t] = (uint16_t)((b + 0x7FFFu + ((b >> 16) & 1u)) >> 16);
    }
}

// label[h][i] = argmax_c <q_i, center_c> (lowest c on ties); hist[h][c] counts
// the labels (a block of 4 waves labels kLabelRounds * 128 queries, then adds
// its 256 counts).  A wave takes 32 queries of one head and scores them against
// 32 centres at a time with one bf16 MFMA per 16 dimensions (A = centres,
// B = queries, so lane l holds the scores of query l % 32); lanes l and
// l + 32 hold different centres of the same query and merge their maxima.
// The labels only decide which queries the select kernel groups together.
constexpr int kLabelRounds = 8;   // rounds of 128 queries per labelling block

template <int D>
__global__ __launch_bounds__(256) void group_label_kernel(const uint16_t* __restrict__ Q,
                                                          const uint16_t* __restrict__ centers,
                                                          int32_t N, int32_t H,
                                                          uint16_t* __restrict__ label,
                                                          int32_t* __restrict__ hist) {
    constexpr int NC = D / 16;
    constexpr int TB = 4;   // the loads of four centre tiles go out together
    static_assert(C % (32 * TB) == 0, "whole groups of centre tiles");
    __shared__ int32_t lh[C];
    const int h = blockIdx.y;
    const int lane = threadIdx.x & 63;
    const int col = lane & 31, half = lane >> 5;
    lh[threadIdx.x] = 0;
    __syncthreads();
    const uint16_t* ch = centers + (size_t)h * C * D + (size_t)col * D + 8 * half;
    for (int rd = 0; rd < kLabelRounds; ++rd) {
        const int64_t i = ((int64_t)blockIdx.x * kLabelRounds + rd) * 128 + (threadIdx.x >> 6) * 32 + col;
        const bool valid = i < N;
        bf16x8 bq[NC];
        const uint16_t* row = Q + ((size_t)(valid ? i : 0) * H + h) * D + 8 * half;
#pragma unroll
        for (int c = 0; c < NC; ++c)
            bq[c] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(row + 16 * c));
        float best = -INFINITY;
        int arg = 0;
        for (int c0 = 0; c0 < C; c0 += 32 * TB) {
            uint4 ct[TB][NC];
#pragma unroll
            for (int tb = 0; tb < TB; ++tb)
#pragma unroll
                for (int c = 0; c < NC; ++c)
                    ct[tb][c] = *reinterpret_cast<const uint4*>(ch + (size_t)(c0 + 32 * tb) * D + 16 * c);
#pragma unroll
            for (int tb = 0; tb < TB; ++tb) {
                f32x16 acc = f32x16{};
#pragma unroll
                for (int c = 0; c < NC; ++c)
                    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, ct[tb][c]), bq[c], acc,
                                                                  0, 0, 0);
                // rows 8 (r / 4) + 4 half + r % 4 increase with r: strict >
                // keeps the lowest centre
                const int cb = c0 + 32 * tb;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int cc = cb + 8 * (r >> 2) + 4 * half + (r & 3);
                    if (acc[r] > best) {
                        best = acc[r];
                        arg = cc;
                    }
                }
            }
        }
        const float ob = __shfl_xor(best, 32);
        const int oa = __shfl_xor(arg, 32);
        if (ob > best || (ob == best && oa < arg)) arg = oa;
        if (valid && half == 0) {
            label[(size_t)h * N + i] = (uint16_t)arg;
            atomicAdd(&lh[arg], 1);
        }
    }
    __syncthreads();
    if (lh[threadIdx.x] != 0) atomicAdd(&hist[(size_t)h * C + threadIdx.x], lh[threadIdx.x]);
}

// Exclusive prefix sum of each head's histogram, in place (one block per head).
__global__ __launch_bounds__(256) void group_scan_kernel(int32_t* __restrict__ hist) {
    __shared__ int32_t s[C];
    int32_t* hh = hist + (size_t)blockIdx.x * C;
    const int t = threadIdx.x;
    const int32_t own = hh[t];
    s[t] = own;
    __syncthreads();
    for (int off = 1; off < C; off <<= 1) {
        const int32_t add = t >= off ? s[t - off] : 0;
        __syncthreads();
        s[t] += add;
        __syncthreads();
    }
    hh[t] = s[t] - own;
}

// perm[h][cursor[h][label]++] = i, for the kScatterPer * 256 queries of a
// block: each query takes its rank among the block's queries of its label
// from an LDS counter, and the block reserves its places with one global
// atomic per label.  The order inside one bucket follows the atomics and is
// not fixed; any order is a valid grouping.
constexpr int kScatterPer = 8;

__global__ __launch_bounds__(256) void group_scatter_kernel(const uint16_t* __restrict__ label,
                                                            int32_t* __restrict__ cursor,
                                                            int32_t N, int32_t H,
                                                            int32_t* __restrict__ perm) {
    __shared__ int32_t cnt[C];
    const int h = blockIdx.y;
    const int t = threadIdx.x;
    const int64_t base = (int64_t)blockIdx.x * 256 * kScatterPer;
    cnt[t] = 0;
    __syncthreads();
    int lab[kScatterPer], rank[kScatterPer];
#pragma unroll
    for (int r = 0; r < kScatterPer; ++r) {
        const int64_t i = base + r * 256 + t;
        lab[r] = i < N ? label[(size_t)h * N + i] : -1;
        rank[r] = lab[r] >= 0 ? atomicAdd(&cnt[lab[r]], 1) : 0;
    }
    __syncthreads();
    const int c = cnt[t];
    if (c != 0) cnt[t] = atomicAdd(&cursor[(size_t)h * C + t], c);
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kScatterPer; ++r) {
        const int64_t i = base + r * 256 + t;
        if (lab[r] >= 0) perm[(size_t)h * N + cnt[lab[r]] + rank[r]] = (int32_t)i;
    }
}

}  // namespace

size_t group_workspace_bytes(int32_t N, int32_t H, int32_t d) {
    auto al = [](size_t x) { return (x + 255) / 256 * 256; };
    return al((size_t)H * C * d * sizeof(uint16_t)) + al((size_t)H * N * sizeof(uint16_t)) +
           al((size_t)2 * H * C * sizeof(int32_t)) + al((size_t)H * N * sizeof(int32_t));
}

const int32_t* group_perm_in(const void* ws, int32_t N, int32_t H, int32_t d) {
    auto al = [](size_t x) { return (x + 255) / 256 * 256; };
    const char* p = reinterpret_cast<const char*>(ws);
    p += al((size_t)H * C * d * sizeof(uint16_t)) + al((size_t)H * N * sizeof(uint16_t)) +
         al((size_t)2 * H * C * sizeof(int32_t));
    return reinterpret_cast<const int32_t*>(p);
}

hipError_t launch_group_queries(const void* Q, int32_t N, int32_t H, int32_t d, void* ws,
                                QueryGroups* out, hipStream_t stream) {
    auto al = [](size_t x) { return (x + 255) / 256 * 256; };
    char* p = reinterpret_cast<char*>(ws);
    uint16_t* centers = reinterpret_cast<uint16_t*>(p);
    p += al((size_t)H * C * d * sizeof(uint16_t));
    uint16_t* label = reinterpret_cast<uint16_t*>(p);
    p += al((size_t)H * N * sizeof(uint16_t));
    int32_t* hist = reinterpret_cast<int32_t*>(p);          // [H][C], then seed_ref [H][C]
    int32_t* seed_ref = hist + (size_t)H * C;
    p += al((size_t)2 * H * C * sizeof(int32_t));
    int32_t* perm = reinterpret_cast<int32_t*>(p);
    out->perm = perm;
    out->label = label;
    out->seed_ref = seed_ref;

    const uint16_t* q = reinterpret_cast<const uint16_t*>(Q);
    hipError_t e = launch_fill_zero(reinterpret_cast<float*>(hist), (size_t)2 * H * C, stream);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(group_centers_kernel, dim3(H), dim3(C), 0, stream, q, N, H, d, centers);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const dim3 grid((unsigned)((N + 128 * kLabelRounds - 1) / (128 * kLabelRounds)), (unsigned)H);
    if (d == 16)
        hipLaunchKernelGGL(group_label_kernel<16>, grid, dim3(256), 0, stream, q, centers, N, H, label, hist);
    else if (d == 32)
        hipLaunchKernelGGL(group_label_kernel<32>, grid, dim3(256), 0, stream, q, centers, N, H, label, hist);
    else if (d == 64)
        hipLaunchKernelGGL(group_label_kernel<64>, grid, dim3(256), 0, stream, q, centers, N, H, label, hist);
    else
        hipLaunchKernelGGL(group_label_kernel<128>, grid, dim3(256), 0, stream, q, centers, N, H, label, hist);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(group_scan_kernel, dim3(H), dim3(C), 0, stream, hist);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const dim3 sgrid((unsigned)((N + 256 * kScatterPer - 1) / (256 * kScatterPer)), (unsigned)H);
    hipLaunchKernelGGL(group_scatter_kernel, sgrid, dim3(256), 0, stream, label, hist, N, H, perm);
    return hipGetLastError();
}

}  // namespace kmip
