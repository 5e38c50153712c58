// Backward of k-MIP attention on gfx950, index set held fixed.
//
// The forward's top-k indices are reused (Section 3.1, last paragraph, and
// Appendix E, last paragraph, of arXiv 2604.03815), so only the k selected
// pairs of each query carry gradient.  With z_j = scale * s_ij recomputed in
// fp32 exactly as the forward aggregate does, p_j = exp(z_j - lse_i):
//   dp_j = dO_i . v_j,  D_i = sum_j p_j dp_j,  g_j = p_j (dp_j - D_i)
//   dQ_i = scale sum_j g_j k_j      (row-local, plain store)
//   dK_j += scale g_j q_i,  dV_j += p_j dO_i   (scatter with fp32 atomics)
//
// Mapping: a team of 16 lanes per (query, head) as in the aggregate kernel:
// slots on lanes for the per-pair scalars, dimensions on lanes for the
// row-vector updates, so each atomic instruction of a team covers one
// contiguous 64-byte run of a dK or dV row.
#include "kmip_device.h"
#include "kmip_internal.h"

namespace kmip {
namespace {

constexpr int kMaxSlotsPerLane = (128 + 15) / 16;

template <int D>
__global__ __launch_bounds__(256) void bwd_atomic_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K, const uint16_t* __restrict__ V,
    const uint16_t* __restrict__ dO, const int32_t* __restrict__ idx, const float* __restrict__ lse,
    int32_t N, int32_t H, int32_t k, float scale, float* __restrict__ dQ, float* __restrict__ dK,
    float* __restrict__ dV) {
    const int tl = threadIdx.x & 15;
    const int64_t qh = (int64_t)blockIdx.x * 16 + (threadIdx.x >> 4);
    if (qh >= (int64_t)N * H) return;  // whole team exits together
    const int h = (int)(qh % H);

    float q[D], g[D];
    load_row_f32<D>(q, Q + (size_t)qh * D);
    load_row_f32<D>(g, dO + (size_t)qh * D);
    const float l = lse[qh];

    const int ns = (k + 15) >> 4;
    float p[kMaxSlotsPerLane], dp[kMaxSlotsPerLane];
    int32_t jj[kMaxSlotsPerLane];
    float dsum = 0.0f;
#pragma unroll
    for (int s = 0; s < kMaxSlotsPerLane; ++s) {
        p[s] = 0.0f;
        dp[s] = 0.0f;
        jj[s] = -1;
        const int slot = tl + 16 * s;
        if (s < ns && slot < k && l != -INFINITY) {
            const int32_t j = idx[(size_t)qh * k + slot];
            if (j >= 0 && j < N) {
                jj[s] = j;
                const float z = scale * dot_row_bf16<D>(q, K + ((size_t)j * H + h) * D);
                p[s] = __expf(z - l);
                dp[s] = dot_row_bf16<D>(g, V + ((size_t)j * H + h) * D);
            }
        }
        dsum = fmaf(p[s], dp[s], dsum);
    }
    dsum = group16_sum(dsum);

    constexpr int U = D / 16;
    float qd[U], gd[U], dq[U];
    {
        // this lane's dimensions of q_i and dO_i, read straight from memory so
        // that no runtime register indexing is needed
        const uint16_t* qrow = Q + (size_t)qh * D + tl;
        const uint16_t* grow = dO + (size_t)qh * D + tl;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            qd[u] = bf16_bits_to_f32(qrow[16 * u]);
            gd[u] = bf16_bits_to_f32(grow[16 * u]);
            dq[u] = 0.0f;
        }
    }
#pragma unroll
    for (int s = 0; s < kMaxSlotsPerLane; ++s) {
        if (s < ns) {
            const float gs_own = p[s] * (dp[s] - dsum);
            for (int src = 0; src < 16; ++src) {
                const int32_t js = __shfl(jj[s], src, 16);
                const float gsv = __shfl(gs_own, src, 16);
                const float ps = __shfl(p[s], src, 16);
                if (js >= 0) {
                    const size_t base = ((size_t)js * H + h) * D + tl;
                    const uint16_t* krow = K + base;
#pragma unroll
                    for (int u = 0; u < U; ++u) {
                        dq[u] = fmaf(gsv, bf16_bits_to_f32(krow[16 * u]), dq[u]);
                        atomicAdd(dK + base + 16 * u, scale * gsv * qd[u]);
                        atomicAdd(dV + base + 16 * u, ps * gd[u]);
                    }
                }
            }
        }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) dQ[(size_t)qh * D + tl + 16 * u] = scale * dq[u];
}

__global__ __launch_bounds__(256) void fill_zero_kernel(float4* __restrict__ p, size_t n4) {
    const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (i < n4) p[i] = make_float4(0.f, 0.f, 0.f, 0.f);
}

}  // namespace

hipError_t launch_fill_zero(float* p, size_t n, hipStream_t stream) {
    // n is a multiple of 16 here (rows of d >= 16 floats), so float4 stores cover it.
    const size_t n4 = n / 4;
    if (n4 == 0) return hipSuccess;
    hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0, stream,
                       reinterpret_cast<float4*>(p), n4);
    return hipGetLastError();
}

hipError_t launch_bwd_atomic(const void* Q, const void* K, const void* V, const void* dO,
                             const int32_t* idx, const float* lse, int32_t N, int32_t H,
                             int32_t d, int32_t k, float scale, float* dQ, float* dK, float* dV,
                             hipStream_t stream) {
    const int64_t nqh = (int64_t)N * H;
    if (nqh == 0) return hipSuccess;
    hipError_t e = launch_fill_zero(dK, (size_t)nqh * d, stream);
    if (e != hipSuccess) return e;
    e = launch_fill_zero(dV, (size_t)nqh * d, stream);
    if (e != hipSuccess) return e;
    const unsigned blocks = (unsigned)((nqh + 15) / 16);
    const uint16_t* q = reinterpret_cast<const uint16_t*>(Q);
    const uint16_t* kk = reinterpret_cast<const uint16_t*>(K);
    const uint16_t* v = reinterpret_cast<const uint16_t*>(V);
    const uint16_t* g = reinterpret_cast<const uint16_t*>(dO);
    switch (d) {
        case 16:
            hipLaunchKernelGGL(bwd_atomic_kernel<16>, dim3(blocks), dim3(256), 0, stream, q, kk, v,
                               g, idx, lse, N, H, k, scale, dQ, dK, dV);
            break;
        case 32:
            hipLaunchKernelGGL(bwd_atomic_kernel<32>, dim3(blocks), dim3(256), 0, stream, q, kk, v,
                               g, idx, lse, N, H, k, scale, dQ, dK, dV);
            break;
        case 64:
            hipLaunchKernelGGL(bwd_atomic_kernel<64>, dim3(blocks), dim3(256), 0, stream, q, kk, v,
                               g, idx, lse, N, H, k, scale, dQ, dK, dV);
            break;
        default:
            return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace kmip
