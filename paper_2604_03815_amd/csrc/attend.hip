// Gather-softmax-aggregate for k-MIP attention on gfx950.
//
// Algorithm 1 (Appendix E) of arXiv 2604.03815 after RowwiseTopK: gather the
// k selected value rows (GatherRows), take a softmax over the k kept scores
// times `scale`, and sum the weighted rows (Einsum nk,nkv->nv).  The kept
// scores are recomputed in fp32 from q_i and the gathered key rows, with the
// same routine the backward uses, so the weights of the two passes agree.
//
// Mapping: a team of 16 lanes per (query, head), 16 teams per workgroup,
// with the key slots on lanes (slot = lane + 16 s, NS slots per lane).  Each
// lane gathers its slots' key rows (D = d_K wide) and forms their scores;
// 16-lane butterflies give the softmax statistics; each lane then adds its
// slots' weighted value rows (DV = d_V wide, gathered in the same round trip
// as the key rows when they fit in 64 registers, else right after) into a
// DV-vector, and a transposed team reduction leaves dimensions tl, tl + 16,
// ... on lane tl.
//
// Attention dropout (keep != nullptr): slot t's weight in the sum is
// multiplied by keep_scale when keep[qh k + t] is nonzero and by 0
// otherwise; the softmax statistics (lse) are those before dropout.
//
// Order: with perm == nullptr, team t of block b takes query-head
// 16 b + t.  With a query order perm [H][N] (the forward's grouping of the
// queries by direction), block (b, h) takes positions 16 b .. 16 b + 15 of
// head h in that order: queries of one group select mostly the same keys,
// so the teams of a workgroup gather the same rows.
#include "kmip_device.h"
#include "kmip_internal.h"

namespace kmip {
namespace {

template <int D, int DV, int NS>
__global__ __launch_bounds__(256) void attend_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K, const uint16_t* __restrict__ V,
    const int32_t* __restrict__ idx, const uint8_t* __restrict__ keep, float keep_scale, int32_t N,
    int32_t H, int32_t k, float scale, const int32_t* __restrict__ perm, float* __restrict__ out,
    float* __restrict__ lse) {
    constexpr bool kKeep = DV / 2 * NS <= 64;
    const int tl = threadIdx.x & 15;
    int64_t qh;
    int h;
    if (perm != nullptr) {
        h = blockIdx.y;
        const int64_t p = (int64_t)blockIdx.x * 16 + (threadIdx.x >> 4);
        if (p >= N) return;  // whole team exits together
        qh = (int64_t)perm[(size_t)h * N + p] * H + h;
    } else {
        qh = (int64_t)blockIdx.x * 16 + (threadIdx.x >> 4);
        if (qh >= (int64_t)N * H) return;  // whole team exits together
        h = (int)(qh % H);
    }

    float q[D];
    load_row_f32<D>(q, Q + (size_t)qh * D);

    float z[NS];
    int32_t jj[NS];
    uint4 vw[kKeep ? NS : 1][DV / 8];
    float zmax = -INFINITY;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        z[s] = -INFINITY;
        jj[s] = -1;
        const int slot = tl + 16 * s;
        if (slot < k) {
            const int32_t j = idx[(size_t)qh * k + slot];
            if (j >= 0 && j < N) {
                jj[s] = j;
                if constexpr (kKeep) load_row_words<DV>(vw[s], V + ((size_t)j * H + h) * DV);
                z[s] = scale * dot_row_bf16<D>(q, K + ((size_t)j * H + h) * D);
            }
        }
        zmax = fmaxf(zmax, z[s]);
    }
    zmax = group16_max(zmax);

    float w[NS];
    float zs = 0.0f;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        w[s] = jj[s] >= 0 ? __expf(z[s] - zmax) : 0.0f;
        zs += w[s];
    }
    zs = group16_sum(zs);
    if (keep != nullptr) {
#pragma unroll
        for (int s = 0; s < NS; ++s)
            if (jj[s] >= 0) w[s] *= keep[(size_t)qh * k + tl + 16 * s] != 0 ? keep_scale : 0.0f;
    }

    float acc[DV];
#pragma unroll
    for (int t = 0; t < DV; ++t) acc[t] = 0.0f;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        if (jj[s] >= 0) {
            uint4 wv[DV / 8];
            if constexpr (kKeep) {
#pragma unroll
                for (int c = 0; c < DV / 8; ++c) wv[c] = vw[s][c];
            } else {
                load_row_words<DV>(wv, V + ((size_t)jj[s] * H + h) * DV);
            }
#pragma unroll
            for (int c = 0; c < DV / 8; ++c) {
                const uint32_t ww[4] = {wv[c].x, wv[c].y, wv[c].z, wv[c].w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    acc[8 * c + 2 * e] = fmaf(w[s], bf16_bits_to_f32(ww[e] & 0xFFFFu), acc[8 * c + 2 * e]);
                    acc[8 * c + 2 * e + 1] = fmaf(w[s], bf16_bits_to_f32(ww[e] >> 16), acc[8 * c + 2 * e + 1]);
                }
            }
        }
    }
    float o[DV / 16];
    team_sum_transpose<DV>(acc, o, tl);

    const bool any = zmax != -INFINITY;
    const float inv = any ? 1.0f / zs : 0.0f;
#pragma unroll
    for (int u = 0; u < DV / 16; ++u) out[(size_t)qh * DV + tl + 16 * u] = o[u] * inv;
    if (tl == 0) lse[qh] = any ? zmax + __logf(zs) : -INFINITY;
}

template <int D, int DV>
void launch_attend_d(dim3 blocks, hipStream_t stream, const uint16_t* q, const uint16_t* kk,
                     const uint16_t* v, const int32_t* idx, const uint8_t* keep, float keep_scale, int32_t N,
                     int32_t H, int32_t k, float scale, const int32_t* perm, float* out, float* lse) {
    const int ns = (k + 15) / 16;
    if (ns <= 1)
        hipLaunchKernelGGL((attend_kernel<D, DV, 1>), dim3(blocks), dim3(256), 0, stream, q, kk, v, idx, keep,
                           keep_scale, N, H, k, scale, perm, out, lse);
    else if (ns <= 2)
        hipLaunchKernelGGL((attend_kernel<D, DV, 2>), dim3(blocks), dim3(256), 0, stream, q, kk, v, idx, keep,
                           keep_scale, N, H, k, scale, perm, out, lse);
    else if (ns <= 4)
        hipLaunchKernelGGL((attend_kernel<D, DV, 4>), dim3(blocks), dim3(256), 0, stream, q, kk, v, idx, keep,
                           keep_scale, N, H, k, scale, perm, out, lse);
    else if (ns <= 8)
        hipLaunchKernelGGL((attend_kernel<D, DV, 8>), dim3(blocks), dim3(256), 0, stream, q, kk, v, idx, keep,
                           keep_scale, N, H, k, scale, perm, out, lse);
    else if constexpr (D <= 64) {
        // k > 128 (d <= 64 only)
        if (ns <= 16)
            hipLaunchKernelGGL((attend_kernel<D, DV, 16>), dim3(blocks), dim3(256), 0, stream, q, kk, v, idx, keep,
                               keep_scale, N, H, k, scale, perm, out, lse);
        else
            hipLaunchKernelGGL((attend_kernel<D, DV, 32>), dim3(blocks), dim3(256), 0, stream, q, kk, v, idx, keep,
                               keep_scale, N, H, k, scale, perm, out, lse);
    }
}

}  // namespace

hipError_t launch_attend(const void* Q, const void* K, const void* V, const int32_t* idx,
                         const uint8_t* keep, float keep_scale, int32_t N, int32_t H, int32_t d, int32_t dv,
                         int32_t k, float scale, const int32_t* perm, float* out, float* lse,
                         hipStream_t stream) {
    const int64_t nqh = (int64_t)N * H;
    if (nqh == 0) return hipSuccess;
    const dim3 blocks = perm != nullptr ? dim3((unsigned)((N + 15) / 16), (unsigned)H)
                                        : dim3((unsigned)((nqh + 15) / 16));
    const uint16_t* q = reinterpret_cast<const uint16_t*>(Q);
    const uint16_t* kk = reinterpret_cast<const uint16_t*>(K);
    const uint16_t* v = reinterpret_cast<const uint16_t*>(V);
#define KMIP_ATTEND_CASE(DD, DVV)                                                              \
    if (d == DD && dv == DVV) {                                                                \
        launch_attend_d<DD, DVV>(blocks, stream, q, kk, v, idx, keep, keep_scale, N, H, k, scale, perm, out, lse); \
        return hipGetLastError();                                                              \
    }
#define KMIP_ATTEND_D(DD) \
    KMIP_ATTEND_CASE(DD, 16) KMIP_ATTEND_CASE(DD, 32) KMIP_ATTEND_CASE(DD, 64) KMIP_ATTEND_CASE(DD, 128)
    KMIP_ATTEND_D(16)
    KMIP_ATTEND_D(32)
    KMIP_ATTEND_D(64)
    KMIP_ATTEND_D(128)
#undef KMIP_ATTEND_D
#undef KMIP_ATTEND_CASE
    return hipErrorInvalidValue;
}

}  // namespace kmip
