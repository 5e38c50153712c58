// Low-precision candidate scoring for the score + select of k-MIP attention
// on gfx950: an int8 MFMA prefilter with a provable bound, then an exact
// re-rank of the candidates with the streaming select kernel's bf16 MFMA.
//
// The operation is RowwiseTopK of Algorithm 1 (Appendix E) of arXiv
// 2604.03815 over one graph (Section 3.1, Eq. 1).  The paper names
// lower-precision scoring (FP16/INT8) on matrix cores as its own next step
// (Appendix, comparison with FlashAttention, closing paragraph); this file
// is that step for one graph and k <= 32, kept exact by a bound.
//
// Quantisation.  Per head, keys share one power-of-two scale s_K (the
// smallest with max|K| / s_K <= 127) and k8_j = round(k_j / s_K), clamped to
// [-127, 127].  Per key, e_j = |k_j - s_K k8_j| and n_j = |s_K k8_j|
// (2-norms); per head their maxima e_max, n_max and k_max = max_j |k_j|.
// Each query gets its own power-of-two scale s_q, q8, e_q = |q - s_q q8|
// and |q|.  Every norm is rounded up.
//
// Bound.  I_j = q8 . k8_j is exact (int32 MFMA).  The dequantised rows have
// the exact product s~_j = s_q s_K I_j, and by Cauchy-Schwarz
// |q . k_j - s~_j| <= |q| e_j + e_q n_j <= E = |q| e_max + e_q n_max.  The
// select kernel's fp32 MFMA score S_j of the bf16 rows differs from q . k_j
// by at most delta = 2 (d + 16) 2^-24 |q| k_max (at most d + 16 roundings
// of partial sums no larger than |q| |k_j|).  So |S_j - s~_j| <= E + delta.
//
// Threshold (first pass over the keys).  The keys fall into 64 groups by
// (tile parity, row in the tile); a lane keeps the largest I of each of its
// query's groups it sees.  If M is the k-th largest of a query's 64 group
// maxima (k <= 32), k distinct keys have I >= M, hence S >= s_q s_K M - E -
// delta, so the query's k-th best score S_(k) is at least that.  A key that
// can be among the k best (S_j >= S_(k), ties included) then has
// s_q s_K I_j >= S_j - E - delta >= s_q s_K M - 2 (E + delta), that is
//     I_j >= T = M - ceil(2 (E + delta) / (s_q s_K)).
//
// Candidates (second pass).  The keys with I_j >= T, listed per query: each
// lane of the query's pair appends its rows to its own half of the query's
// list, at most kPrefilterCap / 2.  By the bound every key of the exact
// top-k is listed (recall 1); a query whose half-list would overflow is
// flagged instead, and its block of 32 queries is re-run by the select
// kernel.
//
// Re-rank.  One wave per query-head forms S_j of its candidates with the
// select kernel's MFMA on the same bf16 operands and in the same chunk
// order (the query replicated over the 32 columns), so the scores are the
// same values, and takes the k best by (score descending, index
// ascending): the select kernel's row, order included.
#include "kmip_device.h"
#include "kmip_internal.h"

namespace kmip {
namespace {

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x16 __attribute__((ext_vector_type(16)));

constexpr int kHalfCap = kPrefilterCap / 2;
// Thresholds never go below this (every |I| is below 127^2 * 128 < 2^21),
// which keeps T - 1 - I free of overflow.
constexpr int32_t kLowT = -(1 << 30);

__device__ __forceinline__ int tile_row(int r, int half) {
    return 8 * (r >> 2) + 4 * half + (r & 3);
}

// Smallest power of two s with m / s <= 127, for finite m >= 0 (1 for m = 0).
__device__ __forceinline__ float pow2_scale(float m) {
    if (!(m > 0.0f)) return 1.0f;
    const float x = m * (1.0f / 127.0f) * (1.0f + 0x1p-20f);   // above m / 127
    uint32_t b = __float_as_uint(x);
    if ((b & 0x7F800000u) == 0u) return 0x1p-126f;            // denormal x: the smallest normal
    if ((b & 0x007FFFFFu) != 0u) b = (b & 0xFF800000u) + 0x00800000u;
    return __uint_as_float(b & 0xFF800000u);
}

// Non-negative float bits order like the floats: atomicMax on them.
__device__ __forceinline__ void max_bits(uint32_t* p, float v) {
    atomicMax(p, __float_as_uint(v));
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) v = fmaxf(v, __shfl_xor(v, m));
    return v;
}

// hstat[h][0] = max |k| bits over the head's key elements.
__global__ __launch_bounds__(256) void i8_absmax_kernel(const uint16_t* __restrict__ K, int32_t N, int32_t H,
                                                        int32_t d, uint32_t* __restrict__ hstat) {
    const int h = blockIdx.y;
    const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
    float m = 0.0f;
    if (j < N) {
        const uint16_t* row = K + ((size_t)j * H + h) * d;
        for (int t = 0; t < d; ++t) m = fmaxf(m, fabsf(bf16_bits_to_f32(row[t])));
    }
    m = wave_max(m);
    if ((threadIdx.x & 63) == 0 && m > 0.0f) max_bits(&hstat[4 * h], m);
}

// Int8 key tiles in the operand order of v_mfma_i32_32x32x32_i8: for head h,
// tile t (32 keys) and chunk c of 32 dims, lane l holds the 16 bytes of key
// 32t + l%32, dims 32c + 16(l/32) .. +16 (dims >= d are zero).  Queries use
// the same order for the B operand, so the k-th byte pairs match whatever
// order the instruction sums them in (the sum is an exact integer).  Also
// the per-head maxima hstat[h][1..3] = e_max, n_max, k_max.
template <int D>
__global__ __launch_bounds__(256) void i8_quant_kernel(const uint16_t* __restrict__ K, int32_t N, int32_t H,
                                                       int32_t ntiles, uint32_t* __restrict__ hstat,
                                                       uint4* __restrict__ kp8) {
    constexpr int NC8 = (D + 31) / 32;
    const int h = blockIdx.y;
    const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
    float e = 0.0f, n = 0.0f, kn = 0.0f;
    if (j < N) {
        const float s = pow2_scale(__uint_as_float(hstat[4 * h]));
        float k[D];
        load_row_f32<D>(k, K + ((size_t)j * H + h) * D);
        int8_t q[NC8 * 32];
#pragma unroll
        for (int t = 0; t < NC8 * 32; ++t) q[t] = 0;
#pragma unroll
        for (int t = 0; t < D; ++t) {
            const float r = fminf(127.0f, fmaxf(-127.0f, rintf(k[t] / s)));
            q[t] = (int8_t)r;
            const float err = k[t] - s * r;   // exact: both sides are short multiples of s's ulp
            e = fmaf(err, err, e);
            n = fmaf(s * r, s * r, n);
            kn = fmaf(k[t], k[t], kn);
        }
        // sums of D squares round at most D times: 2^-16 covers them for D <= 128
        e = sqrtf(e) * (1.0f + 0x1p-16f);
        n = sqrtf(n) * (1.0f + 0x1p-16f);
        kn = sqrtf(kn) * (1.0f + 0x1p-16f);
        const int t = (int)(j >> 5), row = (int)(j & 31);
        uint4* base = kp8 + ((size_t)h * (ntiles + kPadTiles) + t) * NC8 * 64;
#pragma unroll
        for (int c = 0; c < NC8; ++c) {
#pragma unroll
            for (int half = 0; half < 2; ++half) {
                uint32_t w[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int b0 = 32 * c + 16 * half + 4 * u;
                    w[u] = (uint32_t)(uint8_t)q[b0] | ((uint32_t)(uint8_t)q[b0 + 1] << 8) |
                           ((uint32_t)(uint8_t)q[b0 + 2] << 16) | ((uint32_t)(uint8_t)q[b0 + 3] << 24);
                }
                base[c * 64 + row + 32 * half] = make_uint4(w[0], w[1], w[2], w[3]);
            }
        }
    }
    e = wave_max(e);
    n = wave_max(n);
    kn = wave_max(kn);
    if ((threadIdx.x & 63) == 0) {
        if (e > 0.0f) max_bits(&hstat[4 * h + 1], e);
        if (n > 0.0f) max_bits(&hstat[4 * h + 2], n);
        if (kn > 0.0f) max_bits(&hstat[4 * h + 3], kn);
    }
}

// Both passes over the keys for 32 queries of one head (one wave per
// workgroup; blockIdx.x = query block, blockIdx.y = head).  Writes each
// query's candidate lists cand[qh][half][..] and their lengths
// ccount[qh][half] (a length above kHalfCap means overflow).
template <int D>
__global__ __launch_bounds__(64) void i8_scan_kernel(const uint4* __restrict__ kp8, const uint16_t* __restrict__ Q,
                                                     const uint32_t* __restrict__ hstat, int32_t N, int32_t H,
                                                     int32_t k, int32_t ntiles, int32_t* __restrict__ cand,
                                                     int32_t* __restrict__ ccount) {
    constexpr int NC8 = (D + 31) / 32;
    __shared__ int32_t gl[32][65];
    const int lane = threadIdx.x, col = lane & 31, half = lane >> 5;
    const int h = blockIdx.y;
    const int64_t qi = (int64_t)blockIdx.x * 32 + col;
    const bool valid = qi < N;

    // the query's int8 operand, scale and error terms
    float qf[D];
    if (valid) {
        load_row_f32<D>(qf, Q + ((size_t)qi * H + h) * D);
    } else {
#pragma unroll
        for (int t = 0; t < D; ++t) qf[t] = 0.0f;
    }
    float qmax = 0.0f;
#pragma unroll
    for (int t = 0; t < D; ++t) qmax = fmaxf(qmax, fabsf(qf[t]));
    const float sq = pow2_scale(qmax);
    float eq = 0.0f, qn = 0.0f;
    int8_t q8[NC8 * 32];
#pragma unroll
    for (int t = 0; t < NC8 * 32; ++t) q8[t] = 0;
#pragma unroll
    for (int t = 0; t < D; ++t) {
        const float r = fminf(127.0f, fmaxf(-127.0f, rintf(qf[t] / sq)));
        q8[t] = (int8_t)r;
        const float err = qf[t] - sq * r;
        eq = fmaf(err, err, eq);
        qn = fmaf(qf[t], qf[t], qn);
    }
    eq = sqrtf(eq) * (1.0f + 0x1p-16f);
    qn = sqrtf(qn) * (1.0f + 0x1p-16f);
    i32x4 bq[NC8];
#pragma unroll
    for (int c = 0; c < NC8; ++c) {
        int w[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int b0 = 32 * c + 16 * half + 4 * u;
            w[u] = (int)((uint32_t)(uint8_t)q8[b0] | ((uint32_t)(uint8_t)q8[b0 + 1] << 8) |
                         ((uint32_t)(uint8_t)q8[b0 + 2] << 16) | ((uint32_t)(uint8_t)q8[b0 + 3] << 24));
        }
        bq[c] = i32x4{w[0], w[1], w[2], w[3]};
    }
    const float sK = pow2_scale(__uint_as_float(hstat[4 * h]));
    const float emax = __uint_as_float(hstat[4 * h + 1]);
    const float nmax = __uint_as_float(hstat[4 * h + 2]);
    const float kmax = __uint_as_float(hstat[4 * h + 3]);
    const float E = fmaf(qn, emax, eq * nmax) * (1.0f + 0x1p-20f);
    const float delta = 2.0f * (float)(D + 16) * 0x1p-24f * qn * kmax;
    // gap in integer units, rounded up with room for the float arithmetic
    const float gap = 2.0f * (E + delta) / (sq * sK) * (1.0f + 0x1p-10f) + 1.0f;
    const int32_t dT = gap >= 0x1p30f ? (1 << 30) : (int32_t)ceilf(gap);

    // Key tiles stream through a ring of PF tiles in registers, loaded PF
    // tiles ahead.  Tiles past the last one (up to PF - 1 for the rounded
    // loop, PF more for the loads) are the zero padding tiles of the head,
    // and every row at or past N is masked out of the scores.
    constexpr int PF = 4;
    static_assert(2 * PF <= kPadTiles, "prefetches stay inside the padding");
    const uint4* tiles = kp8 + (size_t)h * (ntiles + kPadTiles) * NC8 * 64 + lane;
    const int nt_round = (ntiles + PF - 1) / PF * PF;
    uint4 ring[PF][NC8];
    auto load = [&](uint4 (&slot)[NC8], int t) {
#pragma unroll
        for (int c = 0; c < NC8; ++c) slot[c] = tiles[((size_t)t * NC8 + c) * 64];
    };
    auto score = [&](const uint4 (&slot)[NC8], int t) {
        i32x16 acc = i32x16{};
#pragma unroll
        for (int c = 0; c < NC8; ++c)
            acc = __builtin_amdgcn_mfma_i32_32x32x32_i8(
                i32x4{(int)slot[c].x, (int)slot[c].y, (int)slot[c].z, (int)slot[c].w}, bq[c], acc, 0, 0, 0);
        if (32 * t + 32 > N) {
#pragma unroll
            for (int r = 0; r < 16; ++r)
                if (32 * t + tile_row(r, half) >= N) acc[r] = INT32_MIN;
        }
        return acc;
    };

    // pass 1: group maxima, groups (t & 1, row)
    int32_t gm[2][16];
#pragma unroll
    for (int p = 0; p < 2; ++p)
#pragma unroll
        for (int r = 0; r < 16; ++r) gm[p][r] = INT32_MIN;
#pragma unroll
    for (int u = 0; u < PF; ++u) load(ring[u], u);
    for (int t0 = 0; t0 < nt_round; t0 += PF) {
#pragma unroll
        for (int u = 0; u < PF; ++u) {
            const i32x16 a = score(ring[u], t0 + u);
            load(ring[u], t0 + u + PF);
#pragma unroll
            for (int r = 0; r < 16; ++r) gm[u & 1][r] = max(gm[u & 1][r], a[r]);
        }
    }
#pragma unroll
    for (int p = 0; p < 2; ++p)
#pragma unroll
        for (int r = 0; r < 16; ++r) gl[col][32 * p + tile_row(r, half)] = gm[p][r];
    __syncthreads();
    // M: the k-th largest of the 64 group maxima (ties ranked by position);
    // lane half 'half' ranks groups 32 half .. 32 half + 31
    int32_t M = INT32_MIN;
    for (int g = 32 * half; g < 32 * half + 32; ++g) {
        const int32_t v = gl[col][g];
        int rank = 0;
        for (int f = 0; f < 64; ++f) {
            const int32_t u = gl[col][f];
            rank += (u > v || (u == v && f < g)) ? 1 : 0;
        }
        if (rank == k - 1) M = v;
    }
    M = max(M, __shfl_xor(M, 32));
    const int32_t T = (M == INT32_MIN || M - kLowT <= dT) ? kLowT : M - dT;

    // pass 2: candidates I >= T, into this lane's half of the query's list
    int32_t* mine = cand + ((size_t)(valid ? qi : 0) * H + h) * kPrefilterCap + half * kHalfCap;
    int cnt = 0;
#pragma unroll
    for (int u = 0; u < PF; ++u) load(ring[u], u);
    for (int t0 = 0; t0 < nt_round; t0 += PF) {
#pragma unroll
        for (int u = 0; u < PF; ++u) {
            const int t = t0 + u;
            const i32x16 a = score(ring[u], t);
            load(ring[u], t + PF);
            int32_t m = max(max(max(a[0], a[1]), max(a[2], a[3])), max(max(a[4], a[5]), max(a[6], a[7])));
            m = max(m, max(max(max(a[8], a[9]), max(a[10], a[11])), max(max(a[12], a[13]), max(a[14], a[15]))));
            const bool hit = valid && m >= T;
            if (__builtin_amdgcn_ballot_w64(hit) != 0ull && hit) {
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    if (a[r] >= T) {
                        if (cnt < kHalfCap) mine[cnt] = 32 * t + tile_row(r, half);
                        ++cnt;
                    }
                }
            }
        }
    }
    if (valid) ccount[((size_t)qi * H + h) * 2 + half] = cnt;
}

// Exact re-rank, one wave per query-head qh (blockIdx.x).  Overflowed
// query-heads set the flag of their (head, query block) and write nothing.
template <int D>
__global__ __launch_bounds__(64) void i8_rerank_kernel(const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
                                                       const int32_t* __restrict__ cand,
                                                       const int32_t* __restrict__ ccount, int32_t N, int32_t H,
                                                       int32_t k, int32_t nblocks, int32_t* __restrict__ flags,
                                                       int32_t* __restrict__ topk_idx) {
    constexpr int NC = D / 16;
    constexpr int PER = kPrefilterCap / 64;
    __shared__ float sc[kPrefilterCap];
    __shared__ int32_t ci[kPrefilterCap];
    const int lane = threadIdx.x, col = lane & 31, half = lane >> 5;
    const int64_t qh = blockIdx.x;
    const int64_t qi = qh / H;
    const int h = (int)(qh - qi * H);
    const int c0 = ccount[2 * qh], c1 = ccount[2 * qh + 1];
    if (c0 > kHalfCap || c1 > kHalfCap) {
        if (lane == 0) flags[(size_t)h * nblocks + qi / 32] = 1;
        return;
    }
    const int c = c0 + c1;
    const int32_t* l0 = cand + (size_t)qh * kPrefilterCap;
    const int32_t* l1 = l0 + kHalfCap;
    bf16x8 bq[NC];
    {
        const uint16_t* qrow = Q + (size_t)qh * D + 8 * half;
#pragma unroll
        for (int u = 0; u < NC; ++u) bq[u] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(qrow + 16 * u));
    }
    for (int t0 = 0; t0 < c; t0 += 32) {
        const int e = t0 + col;
        const int32_t j = e < c ? (e < c0 ? l0[e] : l1[e - c0]) : -1;
        const uint4* src = reinterpret_cast<const uint4*>(K + ((size_t)(j >= 0 ? j : 0) * H + h) * D + 8 * half);
        f32x16 acc = f32x16{};
#pragma unroll
        for (int u = 0; u < NC; ++u) {
            const uint4 a = j >= 0 ? src[2 * u] : make_uint4(0, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), bq[u], acc, 0, 0, 0);
        }
        if (half == 0 && e < c) ci[e] = j;
        if (col == 0) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int er = t0 + tile_row(r, half);
                if (er < c) sc[er] = acc[r];
            }
        }
    }
    __syncthreads();
    uint64_t key[PER];
#pragma unroll
    for (int m = 0; m < PER; ++m) {
        const int e = lane + 64 * m;
        key[m] = e < c ? make_key(sc[e], ci[e]) : 0ull;
    }
    int32_t* dst = topk_idx + (size_t)qh * k;
    // registers past the wave-uniform count c hold no key: skipped by a
    // uniform branch rather than compared
    for (int p = 0; p < k; ++p) {
        uint64_t best = key[0];
#pragma unroll
        for (int m = 1; m < PER; ++m)
            if (64 * m < c) best = key[m] > best ? key[m] : best;
#pragma unroll
        for (int s = 32; s >= 1; s >>= 1) {
            const uint64_t o = ((uint64_t)(uint32_t)__shfl_xor((int)(best >> 32), s) << 32) |
                               (uint32_t)__shfl_xor((int)(uint32_t)best, s);
            best = o > best ? o : best;
        }
        if (lane == 0) dst[p] = best == 0ull ? -1 : key_index(best);
#pragma unroll
        for (int m = 0; m < PER; ++m)
            if (64 * m < c) key[m] = key[m] == best ? 0ull : key[m];
    }
}

// Task list of the query blocks with a flag in any head (the rest of the
// list is left as zero-query tasks, which the select kernel skips).
__global__ __launch_bounds__(256) void i8_fallback_tasks_kernel(const int32_t* __restrict__ flags, int32_t nblocks,
                                                                int32_t H, int32_t N, int32_t* __restrict__ count,
                                                                Task* __restrict__ tasks) {
    const int b = blockIdx.x * 256 + threadIdx.x;
    if (b >= nblocks) return;
    bool any = false;
    for (int h = 0; h < H; ++h) any = any || flags[(size_t)h * nblocks + b] != 0;
    if (!any) return;
    const int pos = atomicAdd(count, 1);
    tasks[pos] = Task{32 * b, min(32, N - 32 * b), 0, N};
}

}  // namespace

size_t prefilter_tile_bytes(int32_t N, int32_t H, int32_t d) {
    const size_t ntiles = (size_t)(N + 31) / 32;
    return (size_t)H * (ntiles + kPadTiles) * ((d + 31) / 32) * 64 * 16;
}

hipError_t launch_prefilter(const void* K_, const void* Q_, int32_t N, int32_t H, int32_t d, int32_t k,
                            uint32_t* hstat, uint4* kp8, int32_t* cand, int32_t* ccount, int32_t* flags,
                            int32_t* fb_count, Task* fb_tasks, int32_t* topk_idx, hipStream_t stream) {
    const uint16_t* K = reinterpret_cast<const uint16_t*>(K_);
    const uint16_t* Q = reinterpret_cast<const uint16_t*>(Q_);
    const int32_t ntiles = (N + 31) / 32;
    const int32_t nblocks = ntiles;
    hipError_t e;
    if ((e = launch_fill_zero(reinterpret_cast<float*>(hstat), (size_t)4 * H, stream)) != hipSuccess) return e;
    if ((e = launch_fill_zero(reinterpret_cast<float*>(flags), (size_t)H * nblocks, stream)) != hipSuccess) return e;
    if ((e = launch_fill_zero(reinterpret_cast<float*>(fb_count), 1, stream)) != hipSuccess) return e;
    if ((e = launch_fill_zero(reinterpret_cast<float*>(fb_tasks), (size_t)nblocks * 4, stream)) != hipSuccess)
        return e;
    if ((e = launch_fill_zero(reinterpret_cast<float*>(kp8), prefilter_tile_bytes(N, H, d) / 4, stream)) !=
        hipSuccess)
        return e;
    const dim3 kgrid((unsigned)((N + 255) / 256), (unsigned)H);
    hipLaunchKernelGGL(i8_absmax_kernel, kgrid, dim3(256), 0, stream, K, N, H, d, hstat);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const dim3 sgrid((unsigned)nblocks, (unsigned)H);
    const unsigned rgrid = (unsigned)((int64_t)N * H);
#define KMIP_PREFILTER_D(DD)                                                                                    \
    if (d == DD) {                                                                                              \
        hipLaunchKernelGGL(i8_quant_kernel<DD>, kgrid, dim3(256), 0, stream, K, N, H, ntiles, hstat, kp8);      \
        if ((e = hipGetLastError()) != hipSuccess) return e;                                                    \
        hipLaunchKernelGGL(i8_scan_kernel<DD>, sgrid, dim3(64), 0, stream, kp8, Q, hstat, N, H, k, ntiles, cand, \
                           ccount);                                                                             \
        if ((e = hipGetLastError()) != hipSuccess) return e;                                                    \
        hipLaunchKernelGGL(i8_rerank_kernel<DD>, dim3(rgrid), dim3(64), 0, stream, Q, K, cand, ccount, N, H, k,  \
                           nblocks, flags, topk_idx);                                                           \
        if ((e = hipGetLastError()) != hipSuccess) return e;                                                    \
    } else
    KMIP_PREFILTER_D(16)
    KMIP_PREFILTER_D(32)
    KMIP_PREFILTER_D(64)
    KMIP_PREFILTER_D(128)
    return hipErrorInvalidValue;
#undef KMIP_PREFILTER_D
    hipLaunchKernelGGL(i8_fallback_tasks_kernel, dim3((unsigned)((nblocks + 255) / 256)), dim3(256), 0, stream,
                       flags, nblocks, H, N, fb_count, fb_tasks);
    return hipGetLastError();
}

}  // namespace kmip
