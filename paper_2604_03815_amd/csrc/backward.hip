// Backward of k-MIP attention on gfx950, index set held fixed.
//
// The forward's top-k indices are reused (Section 3.1, last paragraph, and
// Appendix E, last paragraph, of arXiv 2604.03815), so only the k selected
// pairs of each query carry gradient.  With z_j = scale * s_ij recomputed in
// fp32 exactly as the forward aggregate does, p_j = exp(z_j - lse_i):
//   dp_j = dO_i . v_j,  D_i = sum_j p_j dp_j,  g_j = p_j (dp_j - D_i)
//   dQ_i = scale sum_j g_j k_j      (row-local, plain store)
//   dK_j += scale g_j q_i,  dV_j += p_j dO_i   (scatter)
// With attention dropout (keep != nullptr, f_j = keep_scale or 0 by the
// forward's keep draw of slot j), dp_j is replaced by f_j dp_j in D_i and
// g_j, and dV_j gets p_j f_j dO_i.
//
// D is the query/key width d_K, DV the value width d_V (dp_j and dV run over
// DV dimensions, dQ and dK over D).
// Mapping: a team of 16 lanes per (query, head) as in the aggregate kernel:
// slots on lanes for the per-pair scalars, dimensions on lanes for the
// row-vector updates.  Two ways to scatter:
//   * per pair: each pair adds its dK and dV rows with fp32 atomics, one
//     64-byte run per instruction;
//   * key-aggregated: the queries are grouped by direction (group.hip), so
//     the 256 queries of a workgroup share most of their keys; the
//     workgroup sums its pairs per key in an LDS hash table and adds each
//     key's sums to dK and dV with one atomic per dimension.  Pairs whose
//     key finds no table slot add directly.  When a few keys are selected
//     by most queries, per-pair atomics serialise on those keys' rows; the
//     table removes nearly all of them.
#include "kmip_device.h"
#include "kmip_internal.h"

namespace kmip {
namespace {

// Key-aggregated scatter: a workgroup of 16 teams takes kAggQueries
// consecutive positions of one head in the grouped query order, and sums
// per key in a table of kSlots keys (32 KB of sums).
constexpr int kAggQueries = 256;

template <int D, int DV>
struct AggTable {
    // the largest power of two with kSlots (D + DV) floats <= 32 KB
    static constexpr int kSlots = D + DV <= 32 ? 256 : D + DV <= 64 ? 128 : D + DV <= 128 ? 64 : 32;
    static constexpr int kProbes = 8;
};

// LDS table of one workgroup: key row index and the D + DV sums (dK, then dV).
template <int D, int DV>
struct AggLds {
    int32_t key[AggTable<D, DV>::kSlots];
    float acc[AggTable<D, DV>::kSlots][D + DV];
};

// Finds or claims the table slot of key row js; -1 when all probes are taken
// by other keys.  A plain read finds a key that is in the table already (the
// common case, and a broadcast when many lanes ask for the same key); only an
// empty slot is claimed with a compare-and-swap.  Every lane of a team runs
// the same probes, and a claim by one of them reads back as the key itself
// for the others.
template <int D, int DV>
__device__ __forceinline__ int agg_slot(AggLds<D, DV>* t, int32_t js) {
    constexpr int C = AggTable<D, DV>::kSlots;
    const uint32_t hsh = ((uint32_t)js * 0x9E3779B1u) >> (32 - __builtin_ctz(C));
    for (int p = 0; p < AggTable<D, DV>::kProbes; ++p) {
        const int ts = (int)((hsh + p) & (C - 1));
        const int32_t cur = __hip_atomic_load(&t->key[ts], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        if (cur == js) return ts;
        if (cur == -1) {
            const int32_t old = atomicCAS(&t->key[ts], -1, js);
            if (old == -1 || old == js) return ts;
        }
    }
    return -1;
}

// Backward of one (query, head) qh by a team of 16 lanes (tl = lane in team).
// Pair scalars live with the slots on lanes; for the scatter, each round of
// 16 slots is broadcast to the team, which then works with dimensions on
// lanes.  All 16 pairs' key elements for dQ are loaded before any is used.
// With tab != nullptr the dK/dV sums go to the workgroup's table when the
// key has a slot there.  MS: slots per lane the registers hold (k <= 16 MS).
template <int D, int DV, int MS>
__device__ __forceinline__ void bwd_query(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K, const uint16_t* __restrict__ V,
    const uint16_t* __restrict__ dO, const int32_t* __restrict__ idx, const float* __restrict__ lse,
    const uint8_t* __restrict__ keep, float keep_scale, int64_t qh, int h, int tl, int32_t N, int32_t H,
    int32_t k, float scale, float* __restrict__ dQ, float* __restrict__ dK, float* __restrict__ dV,
    AggLds<D, DV>* tab) {
    constexpr int U = D / 16;
    constexpr int UV = DV / 16;
    float q[D], g[DV];
    load_row_f32<D>(q, Q + (size_t)qh * D);
    load_row_f32<DV>(g, dO + (size_t)qh * DV);
    const float l = lse[qh];

    const int ns = (k + 15) >> 4;
    float p[MS], dp[MS], pv[MS];
    int32_t jj[MS];
    float dsum = 0.0f;
#pragma unroll
    for (int s = 0; s < MS; ++s) {
        p[s] = 0.0f;
        dp[s] = 0.0f;
        pv[s] = 0.0f;
        jj[s] = -1;
        const int slot = tl + 16 * s;
        if (s < ns && slot < k && l != -INFINITY) {
            const int32_t j = idx[(size_t)qh * k + slot];
            if (j >= 0 && j < N) {
                jj[s] = j;
                const float z = scale * dot_row_bf16<D>(q, K + ((size_t)j * H + h) * D);
                p[s] = __expf(z - l);
                dp[s] = dot_row_bf16<DV>(g, V + ((size_t)j * H + h) * DV);
                pv[s] = p[s];
                if (keep != nullptr) {
                    // dropout: the gradient of p_j is f_j dp_j, and dV_j takes p_j f_j
                    const float f = keep[(size_t)qh * k + slot] != 0 ? keep_scale : 0.0f;
                    dp[s] *= f;
                    pv[s] = p[s] * f;
                }
            }
        }
        dsum = fmaf(p[s], dp[s], dsum);
    }
    dsum = group16_sum(dsum);

    float qd[U], gd[UV], dq[U];
    {
        // this lane's dimensions of q_i and dO_i, read straight from memory so
        // that no runtime register indexing is needed
        const uint16_t* qrow = Q + (size_t)qh * D + tl;
        const uint16_t* grow = dO + (size_t)qh * DV + tl;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            qd[u] = bf16_bits_to_f32(qrow[16 * u]);
            dq[u] = 0.0f;
        }
#pragma unroll
        for (int u = 0; u < UV; ++u) gd[u] = bf16_bits_to_f32(grow[16 * u]);
    }
#pragma unroll
    for (int s = 0; s < MS; ++s) {
        if (s < ns) {
            const float gs_own = p[s] * (dp[s] - dsum);
            int32_t js[16];
            float gsv[16], ps[16], kel[16][U];
#pragma unroll
            for (int src = 0; src < 16; ++src) {
                js[src] = __shfl(jj[s], src, 16);
                gsv[src] = __shfl(gs_own, src, 16);
                ps[src] = __shfl(pv[s], src, 16);
            }
#pragma unroll
            for (int src = 0; src < 16; ++src) {
                const uint16_t* krow = K + ((size_t)(js[src] < 0 ? 0 : js[src]) * H + h) * D + tl;
#pragma unroll
                for (int u = 0; u < U; ++u) kel[src][u] = js[src] < 0 ? 0.0f : bf16_bits_to_f32(krow[16 * u]);
            }
#pragma unroll
            for (int src = 0; src < 16; ++src) {
                if (js[src] < 0) continue;
                const int ts = tab != nullptr ? agg_slot<D, DV>(tab, js[src]) : -1;
                if (ts >= 0) {
#pragma unroll
                    for (int u = 0; u < U; ++u) atomicAdd(&tab->acc[ts][16 * u + tl], scale * gsv[src] * qd[u]);
#pragma unroll
                    for (int u = 0; u < UV; ++u) atomicAdd(&tab->acc[ts][D + 16 * u + tl], ps[src] * gd[u]);
                } else {
                    const size_t base = ((size_t)js[src] * H + h) * D + tl;
                    const size_t basev = ((size_t)js[src] * H + h) * DV + tl;
#pragma unroll
                    for (int u = 0; u < U; ++u) atomicAdd(dK + base + 16 * u, scale * gsv[src] * qd[u]);
#pragma unroll
                    for (int u = 0; u < UV; ++u) atomicAdd(dV + basev + 16 * u, ps[src] * gd[u]);
                }
            }
#pragma unroll
            for (int src = 0; src < 16; ++src)
#pragma unroll
                for (int u = 0; u < U; ++u) dq[u] = fmaf(gsv[src], kel[src][u], dq[u]);
        }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) dQ[(size_t)qh * D + tl + 16 * u] = scale * dq[u];
}

// Per-pair scatter: one team per (query, head), 16 per workgroup.
template <int D, int DV, int MS>
__global__ __launch_bounds__(256) void bwd_atomic_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K, const uint16_t* __restrict__ V,
    const uint16_t* __restrict__ dO, const int32_t* __restrict__ idx, const float* __restrict__ lse,
    int32_t N, int32_t H, int32_t k, float scale, float* __restrict__ dQ, float* __restrict__ dK,
    float* __restrict__ dV, const uint8_t* __restrict__ keep, float keep_scale) {
    const int tl = threadIdx.x & 15;
    const int64_t qh = (int64_t)blockIdx.x * 16 + (threadIdx.x >> 4);
    if (qh >= (int64_t)N * H) return;  // whole team exits together
    bwd_query<D, DV, MS>(Q, K, V, dO, idx, lse, keep, keep_scale, qh, (int)(qh % H), tl, N, H, k, scale, dQ, dK,
                         dV, nullptr);
}

// Key-aggregated scatter: one workgroup per kAggQueries positions of head
// blockIdx.y in the grouped order.
template <int D, int DV, int MS>
__global__ __launch_bounds__(256) void bwd_agg_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K, const uint16_t* __restrict__ V,
    const uint16_t* __restrict__ dO, const int32_t* __restrict__ idx, const float* __restrict__ lse,
    const int32_t* __restrict__ perm, int32_t N, int32_t H, int32_t k, float scale,
    float* __restrict__ dQ, float* __restrict__ dK, float* __restrict__ dV, const uint8_t* __restrict__ keep,
    float keep_scale) {
    constexpr int C = AggTable<D, DV>::kSlots;
    constexpr int W = D + DV;
    __shared__ AggLds<D, DV> tab;
    const int tl = threadIdx.x & 15;
    const int team = threadIdx.x >> 4;
    const int h = blockIdx.y;
    for (int e = threadIdx.x; e < C; e += 256) tab.key[e] = -1;
    for (int e = threadIdx.x; e < C * W; e += 256) (&tab.acc[0][0])[e] = 0.0f;
    __syncthreads();
    for (int round = 0; round < kAggQueries / 16; ++round) {
        const int64_t pos = (int64_t)blockIdx.x * kAggQueries + round * 16 + team;
        if (pos >= N) break;  // positions grow with round: the team is done
        const int64_t qh = (int64_t)perm[(size_t)h * N + pos] * H + h;
        bwd_query<D, DV, MS>(Q, K, V, dO, idx, lse, keep, keep_scale, qh, h, tl, N, H, k, scale, dQ, dK, dV, &tab);
    }
    __syncthreads();
    for (int e = threadIdx.x; e < C * W; e += 256) {
        const int s = e / W, c = e - s * W;
        const int32_t j = tab.key[s];
        const float v = (&tab.acc[0][0])[e];
        if (j >= 0 && v != 0.0f) {
            if (c < D)
                atomicAdd(dK + ((size_t)j * H + h) * D + c, v);
            else
                atomicAdd(dV + ((size_t)j * H + h) * DV + (c - D), v);
        }
    }
}

// Zeroes p[0 .. n): a float4 store per thread where four elements remain,
// single stores for a tail of one to three (p is 16-byte aligned).
__global__ __launch_bounds__(256) void fill_zero_kernel(float* __restrict__ p, size_t n) {
    const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
    const size_t e = 4 * i;
    if (e + 4 <= n) {
        reinterpret_cast<float4*>(p)[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    } else {
        for (size_t j = e; j < n; ++j) p[j] = 0.0f;
    }
}

}  // namespace

hipError_t launch_fill_zero(float* p, size_t n, hipStream_t stream) {
    if (n == 0) return hipSuccess;
    const size_t n4 = (n + 3) / 4;
    hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0, stream, p, n);
    return hipGetLastError();
}

hipError_t launch_bwd_atomic(const void* Q, const void* K, const void* V, const void* dO,
                             const int32_t* idx, const float* lse, const uint8_t* keep, float keep_scale,
                             int32_t N, int32_t H, int32_t d, int32_t dv, int32_t k, float scale, float* dQ,
                             float* dK, float* dV, hipStream_t stream) {
    const int64_t nqh = (int64_t)N * H;
    if (nqh == 0) return hipSuccess;
    hipError_t e = launch_fill_zero(dK, (size_t)nqh * d, stream);
    if (e != hipSuccess) return e;
    e = launch_fill_zero(dV, (size_t)nqh * dv, stream);
    if (e != hipSuccess) return e;
    const unsigned blocks = (unsigned)((nqh + 15) / 16);
    const uint16_t* q = reinterpret_cast<const uint16_t*>(Q);
    const uint16_t* kk = reinterpret_cast<const uint16_t*>(K);
    const uint16_t* v = reinterpret_cast<const uint16_t*>(V);
    const uint16_t* g = reinterpret_cast<const uint16_t*>(dO);
    // slots per lane: 8 up to k = 128, 32 beyond (d <= 64 only)
#define KMIP_BWD_ATOMIC_MS(DD, DVV, MSS)                                                                  \
    hipLaunchKernelGGL((bwd_atomic_kernel<DD, DVV, MSS>), dim3(blocks), dim3(256), 0, stream, q, kk, v, g, \
                       idx, lse, N, H, k, scale, dQ, dK, dV, keep, keep_scale);
#define KMIP_BWD_ATOMIC_CASE(DD, DVV)                    \
    if (d == DD && dv == DVV) {                          \
        if (k <= 128 || DD == 128) {                     \
            KMIP_BWD_ATOMIC_MS(DD, DVV, 8)               \
        } else {                                         \
            KMIP_BWD_ATOMIC_MS(DD, DVV, (DD == 128 ? 8 : 32)) \
        }                                                \
        return hipGetLastError();                        \
    }
#define KMIP_BWD_ATOMIC_D(DD) \
    KMIP_BWD_ATOMIC_CASE(DD, 16) KMIP_BWD_ATOMIC_CASE(DD, 32) KMIP_BWD_ATOMIC_CASE(DD, 64) KMIP_BWD_ATOMIC_CASE(DD, 128)
    KMIP_BWD_ATOMIC_D(16)
    KMIP_BWD_ATOMIC_D(32)
    KMIP_BWD_ATOMIC_D(64)
    KMIP_BWD_ATOMIC_D(128)
#undef KMIP_BWD_ATOMIC_MS
#undef KMIP_BWD_ATOMIC_D
#undef KMIP_BWD_ATOMIC_CASE
    return hipErrorInvalidValue;
}

}  // namespace kmip

namespace kmip {

size_t bwd_agg_workspace_bytes(int32_t N, int32_t H, int32_t d) { return group_workspace_bytes(N, H, d); }

hipError_t launch_bwd_agg(const void* Q, const void* K, const void* V, const void* dO,
                          const int32_t* idx, const float* lse, const uint8_t* keep, float keep_scale,
                          int32_t N, int32_t H, int32_t d, int32_t dv, int32_t k, float scale, float* dQ,
                          float* dK, float* dV, void* ws, hipStream_t stream) {
    const int64_t nqh = (int64_t)N * H;
    if (nqh == 0) return hipSuccess;
    QueryGroups groups{};
    hipError_t e = launch_group_queries(Q, N, H, d, ws, &groups, stream);
    if (e != hipSuccess) return e;
    if ((e = launch_fill_zero(dK, (size_t)nqh * d, stream)) != hipSuccess) return e;
    if ((e = launch_fill_zero(dV, (size_t)nqh * dv, stream)) != hipSuccess) return e;
    const dim3 grid((unsigned)((N + kAggQueries - 1) / kAggQueries), (unsigned)H);
    const uint16_t* q = reinterpret_cast<const uint16_t*>(Q);
    const uint16_t* kk = reinterpret_cast<const uint16_t*>(K);
    const uint16_t* v = reinterpret_cast<const uint16_t*>(V);
    const uint16_t* g = reinterpret_cast<const uint16_t*>(dO);
#define KMIP_BWD_AGG_MS(DD, DVV, MSS)                                                                         \
    hipLaunchKernelGGL((bwd_agg_kernel<DD, DVV, MSS>), grid, dim3(256), 0, stream, q, kk, v, g, idx, lse,    \
                       groups.perm, N, H, k, scale, dQ, dK, dV, keep, keep_scale);
#define KMIP_BWD_AGG_CASE(DD, DVV)                     \
    if (d == DD && dv == DVV) {                        \
        if (k <= 128 || DD == 128) {                   \
            KMIP_BWD_AGG_MS(DD, DVV, 8)                \
        } else {                                       \
            KMIP_BWD_AGG_MS(DD, DVV, (DD == 128 ? 8 : 32)) \
        }                                              \
        return hipGetLastError();                      \
    }
#define KMIP_BWD_AGG_D(DD) \
    KMIP_BWD_AGG_CASE(DD, 16) KMIP_BWD_AGG_CASE(DD, 32) KMIP_BWD_AGG_CASE(DD, 64) KMIP_BWD_AGG_CASE(DD, 128)
    KMIP_BWD_AGG_D(16)
    KMIP_BWD_AGG_D(32)
    KMIP_BWD_AGG_D(64)
    KMIP_BWD_AGG_D(128)
#undef KMIP_BWD_AGG_MS
#undef KMIP_BWD_AGG_D
#undef KMIP_BWD_AGG_CASE
    return hipErrorInvalidValue;
}

}  // namespace kmip
