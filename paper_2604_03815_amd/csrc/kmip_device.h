// Device-side helpers shared by the kmip kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kmip {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t bits16) {
    return __uint_as_float(bits16 << 16);
}

// Order-preserving map of a float32 score to uint32 (larger score, larger
// code).  -0 is folded onto +0 first so that equal scores compare equal.
__device__ __forceinline__ uint32_t score_code(float s) {
    uint32_t b = __float_as_uint(s + 0.0f);
    return b ^ ((uint32_t)((int32_t)b >> 31) | 0x80000000u);
}

__device__ __forceinline__ float score_from_code(uint32_t u) {
    uint32_t b = (u & 0x80000000u) ? (u ^ 0x80000000u) : ~u;
    return __uint_as_float(b);
}

// 64-bit selection key: score code in the high word, bitwise-not of the key
// index in the low word.  Larger key = better (higher score, then lower index).
// Key 0 is a sentinel below every real key and decodes to index -1.
__device__ __forceinline__ uint64_t make_key(float s, int32_t j) {
    return ((uint64_t)score_code(s) << 32) | (uint32_t)(~j);
}

__device__ __forceinline__ int32_t key_index(uint64_t key) {
    return ~(int32_t)(uint32_t)key;
}

__device__ __forceinline__ float key_score(uint64_t key) {
    return score_from_code((uint32_t)(key >> 32));
}

// A bf16 row of D values as D/8 16-byte words.
template <int D>
__device__ __forceinline__ void load_row_words(uint4 (&w)[D / 8], const uint16_t* __restrict__ row) {
#pragma unroll
    for (int c = 0; c < D / 8; ++c) w[c] = *reinterpret_cast<const uint4*>(row + 8 * c);
}

// Dot product of a float32 query row held in registers with a bf16 row,
// accumulated in float32 in dimension order t = 0..D-1.  The aggregate and
// the backward kernels both go through this one function, so they see
// bit-identical scores.
template <int D>
__device__ __forceinline__ float dot_words_bf16(const float (&q)[D], const uint4 (&wv)[D / 8]) {
    float s = 0.0f;
#pragma unroll
    for (int c = 0; c < D / 8; ++c) {
        const uint4 u = wv[c];
        uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            s = fmaf(q[8 * c + 2 * e], bf16_bits_to_f32(w[e] & 0xFFFFu), s);
            s = fmaf(q[8 * c + 2 * e + 1], bf16_bits_to_f32(w[e] >> 16), s);
        }
    }
    return s;
}

template <int D>
__device__ __forceinline__ float dot_row_bf16(const float (&q)[D], const uint16_t* __restrict__ row) {
    uint4 w[D / 8];
    load_row_words<D>(w, row);
    return dot_words_bf16<D>(q, w);
}

template <int D>
__device__ __forceinline__ void load_row_f32(float (&q)[D], const uint16_t* __restrict__ row) {
#pragma unroll
    for (int c = 0; c < D / 8; ++c) {
        uint4 u = *reinterpret_cast<const uint4*>(row + 8 * c);
        uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            q[8 * c + 2 * e] = bf16_bits_to_f32(w[e] & 0xFFFFu);
            q[8 * c + 2 * e + 1] = bf16_bits_to_f32(w[e] >> 16);
        }
    }
}

// Reductions over aligned groups of 16 lanes.  A group is one DPP row, so
// the exchanges are DPP row permutes (a modifier of the VALU instruction)
// rather than LDS permutes: row_mirror pairs lane i with 15 - i,
// row_half_mirror with 7 - i (within each half), and the quad permutes with
// i ^ 2 and i ^ 1.  Each of these pairs lanes that differ in the bit of the
// step (8, 4, 2, 1) and agree in every higher bit, which is all a butterfly
// needs.
template <int CTRL>
__device__ __forceinline__ float row_perm(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}

constexpr int kDppRowMirror = 0x140;
constexpr int kDppRowHalfMirror = 0x141;
constexpr int kDppQuadSwap2 = 0x4E;   // quad_perm [2, 3, 0, 1]
constexpr int kDppQuadSwap1 = 0xB1;   // quad_perm [1, 0, 3, 2]

// The partner of the butterfly step with bit m (8, 4, 2, 1).
template <int M>
__device__ __forceinline__ float step_partner(float v) {
    static_assert(M == 8 || M == 4 || M == 2 || M == 1, "steps of a 16-lane group");
    return row_perm<M == 8 ? kDppRowMirror : M == 4 ? kDppRowHalfMirror : M == 2 ? kDppQuadSwap2 : kDppQuadSwap1>(v);
}

__device__ __forceinline__ float group16_max(float v) {
    v = fmaxf(v, step_partner<8>(v));
    v = fmaxf(v, step_partner<4>(v));
    v = fmaxf(v, step_partner<2>(v));
    v = fmaxf(v, step_partner<1>(v));
    return v;
}

__device__ __forceinline__ float group16_sum(float v) {
    v += step_partner<8>(v);
    v += step_partner<4>(v);
    v += step_partner<2>(v);
    v += step_partner<1>(v);
    return v;
}

// Sum of a D-vector over the 16 lanes of a team, transposed: out[u] of lane
// tl receives the team sum of dimension 16u + tl.  Recursive halving: at the
// step with bit m (m = 8, 4, 2, 1) a lane keeps the half of its dimensions
// whose bit m matches its own and adds its partner's values of that half
// (the partner has the other bit m and the same higher bits, so it kept the
// same dimensions so far), so the step exchanges half of what is left (15
// exchanges per 16 dimensions, against 64 for a full butterfly per
// dimension).
template <int N, int M>
__device__ __forceinline__ void halve_step(const float* in, float* outv, int tl) {
    const bool hi = (tl & M) != 0;
#pragma unroll
    for (int b = 0; b < N; b += 2 * M) {
#pragma unroll
        for (int j = 0; j < M; ++j) {
            const float lo_v = in[b + j], hi_v = in[b + M + j];
            const float own = hi ? hi_v : lo_v, other = hi ? lo_v : hi_v;
            outv[b / 2 + j] = own + step_partner<M>(other);
        }
    }
}

template <int D>
__device__ __forceinline__ void team_sum_transpose(const float (&acc)[D], float (&out)[D / 16], int tl) {
    float a8[D / 2], a4[D / 4], a2[D / 8];
    halve_step<D, 8>(acc, a8, tl);
    halve_step<D / 2, 4>(a8, a4, tl);
    halve_step<D / 4, 2>(a4, a2, tl);
    halve_step<D / 8, 1>(a2, out, tl);
}

}  // namespace kmip
