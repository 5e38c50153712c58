// Gather-softmax-aggregate for k-MIP attention on gfx950.
//
// Algorithm 1 (Appendix E) of arXiv 2604.03815 after RowwiseTopK: gather the
// k selected value rows (GatherRows), take a softmax over the k kept scores
// times `scale`, and sum the weighted rows (Einsum nk,nkv->nv).  The kept
// scores are recomputed in fp32 from q_i and the gathered key rows, with the
// same routine the backward uses, so the weights of the two passes agree.
//
// Mapping: a team of 16 lanes per (query, head), 16 teams per workgroup.
// Phase 1 puts key slots on lanes (slot = lane + 16 s) to form the scores and
// the softmax statistics with 16-lane butterflies; phase 2 puts output
// dimensions on lanes (dim = lane + 16 u) and walks the slots, so each team
// reads a gathered value row as one contiguous segment.
#include "kmip_device.h"
#include "kmip_internal.h"

namespace kmip {
namespace {

constexpr int kMaxSlotsPerLane = (128 + 15) / 16;

template <int D>
__global__ __launch_bounds__(256) void attend_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K, const uint16_t* __restrict__ V,
    const int32_t* __restrict__ idx, int32_t N, int32_t H, int32_t k, float scale,
    float* __restrict__ out, float* __restrict__ lse) {
    const int tl = threadIdx.x & 15;
    const int64_t qh = (int64_t)blockIdx.x * 16 + (threadIdx.x >> 4);
    if (qh >= (int64_t)N * H) return;  // whole team exits together
    const int h = (int)(qh % H);

    float q[D];
    load_row_f32<D>(q, Q + (size_t)qh * D);

    const int ns = (k + 15) >> 4;
    float z[kMaxSlotsPerLane];
    int32_t jj[kMaxSlotsPerLane];
    float zmax = -INFINITY;
#pragma unroll
    for (int s = 0; s < kMaxSlotsPerLane; ++s) {
        z[s] = -INFINITY;
        jj[s] = -1;
        const int slot = tl + 16 * s;
        if (s < ns && slot < k) {
            const int32_t j = idx[(size_t)qh * k + slot];
            if (j >= 0 && j < N) {
                jj[s] = j;
                z[s] = scale * dot_row_bf16<D>(q, K + ((size_t)j * H + h) * D);
            }
        }
        zmax = fmaxf(zmax, z[s]);
    }
    zmax = group16_max(zmax);

    float w[kMaxSlotsPerLane];
    float zs = 0.0f;
#pragma unroll
    for (int s = 0; s < kMaxSlotsPerLane; ++s) {
        w[s] = jj[s] >= 0 ? __expf(z[s] - zmax) : 0.0f;
        zs += w[s];
    }
    zs = group16_sum(zs);

    constexpr int U = D / 16;
    float o[U];
#pragma unroll
    for (int u = 0; u < U; ++u) o[u] = 0.0f;
#pragma unroll
    for (int s = 0; s < kMaxSlotsPerLane; ++s) {
        if (s < ns) {
            for (int src = 0; src < 16; ++src) {
                const float ws = __shfl(w[s], src, 16);
                const int32_t js = __shfl(jj[s], src, 16);
                if (js >= 0) {
                    const uint16_t* vrow = V + ((size_t)js * H + h) * D + tl;
#pragma unroll
                    for (int u = 0; u < U; ++u) o[u] = fmaf(ws, bf16_bits_to_f32(vrow[16 * u]), o[u]);
                }
            }
        }
    }

    const bool any = zmax != -INFINITY;
    const float inv = any ? 1.0f / zs : 0.0f;
#pragma unroll
    for (int u = 0; u < U; ++u) out[(size_t)qh * D + tl + 16 * u] = o[u] * inv;
    if (tl == 0) lse[qh] = any ? zmax + __logf(zs) : -INFINITY;
}

}  // namespace

hipError_t launch_attend(const void* Q, const void* K, const void* V, const int32_t* idx,
                         int32_t N, int32_t H, int32_t d, int32_t k, float scale, float* out,
                         float* lse, hipStream_t stream) {
    const int64_t nqh = (int64_t)N * H;
    if (nqh == 0) return hipSuccess;
    const unsigned blocks = (unsigned)((nqh + 15) / 16);
    const uint16_t* q = reinterpret_cast<const uint16_t*>(Q);
    const uint16_t* kk = reinterpret_cast<const uint16_t*>(K);
    const uint16_t* v = reinterpret_cast<const uint16_t*>(V);
    switch (d) {
        case 16:
            hipLaunchKernelGGL(attend_kernel<16>, dim3(blocks), dim3(256), 0, stream, q, kk, v, idx,
                               N, H, k, scale, out, lse);
            break;
        case 32:
            hipLaunchKernelGGL(attend_kernel<32>, dim3(blocks), dim3(256), 0, stream, q, kk, v, idx,
                               N, H, k, scale, out, lse);
            break;
        case 64:
            hipLaunchKernelGGL(attend_kernel<64>, dim3(blocks), dim3(256), 0, stream, q, kk, v, idx,
                               N, H, k, scale, out, lse);
            break;
        default:
            return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace kmip
