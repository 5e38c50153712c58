// Backward of k-MIP attention with a key-sorted segmented reduction.
//
// Same gradients as backward.hip (index set held fixed; Section 3.1, last
// paragraph, and Appendix E, last paragraph, of arXiv 2604.03815):
//   dQ_i = scale sum_j g_ij k_j,  dK_j = sum_i a_ij q_i,  dV_j = sum_i p_ij dO_i
// with a_ij = scale g_ij.  Instead of scattering every pair's rows with
// atomics, the pairs are sorted by key (a counting sort on the key row
// j*H + h), and each key's rows are summed in registers over its run:
//   1. coef:   per (query, head): p, dp, D, g; dQ_i; coefficients (a, p) of
//              each selected pair, stored in pair order;
//   2. count:  pairs per key row;
//   3. scan:   exclusive prefix sum of the counts (three small kernels);
//   4. place:  the pairs' records (key row, query, coefficients) in key
//              order (the scanned counts serve as cursors);
//   5. reduce: fixed chunks of the sorted pairs; a team of 16 lanes walks a
//              contiguous stretch, dimensions on lanes, keeps the running
//              sums of the current key in registers and adds them to dK and
//              dV with one atomic per dimension where the key changes or
//              the stretch ends.
// Counting and placing aggregate equal key rows within a workgroup of 256
// queries first, so a key that most queries select costs one global atomic
// per workgroup, not one per pair.
#include "kmip_device.h"
#include "kmip_internal.h"

#include <algorithm>
#include <type_traits>

namespace kmip {
namespace {

constexpr int kScanBlock = 1024;     // counts per block of the scan
constexpr int kChunk = 1024;         // sorted pairs per wave in the reduction

// 1. Per (query, head), a team of 16 lanes with the slots on lanes, NS
// slots per lane (k <= 16 NS): p, dp, D, g of each selected pair, dQ_i, and
// (QGt != nullptr, value width DV = D only) row qg_row of the interleaved
// copy of q_i and dO_i.  D is the query/key width, DV the value width (dp_j runs
// over it).  Slot tl + 16 s of query-head qh leaves its key index in jj[s]
// (-1: none) and its coefficients a = scale g, p in ca[s], cp[s].  With
// attention dropout (keep != nullptr, f = keep_scale or 0 by the slot's keep
// draw) dp is replaced by f dp and the dV coefficient is p f.
template <int D, int DV, int NS>
__device__ __forceinline__ void coef_one(const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
                                         const uint16_t* __restrict__ V, const uint16_t* __restrict__ dO,
                                         const int32_t* __restrict__ idx, const float* __restrict__ lse,
                                         const uint8_t* __restrict__ keep, float keep_scale,
                                         int32_t N, int32_t H, int32_t k, float scale, int64_t qh, int tl,
                                         float* __restrict__ dQ, uint16_t* __restrict__ QGt, size_t qg_row,
                                         int32_t (&jj)[NS],
                                         float (&ca)[NS], float (&cp)[NS]) {
    // key rows kept in registers for dQ when they take at most 64 dwords a
    // lane; otherwise read again (from cache)
    constexpr bool kKeep = D / 2 * NS <= 64;
    const int h = (int)(qh % H);
    if (DV == D && QGt != nullptr && tl < D / 4) {
        // interleaved copy: row qg_row holds q_i then dO_i, so the reduction
        // gathers both with one load
        const uint16_t* src = tl < D / 8 ? Q + (size_t)qh * D : dO + (size_t)qh * D;
        reinterpret_cast<uint4*>(QGt + qg_row * (2 * D))[tl] = reinterpret_cast<const uint4*>(src)[tl & (D / 8 - 1)];
    }
    float q[D], g[DV];
    load_row_f32<D>(q, Q + (size_t)qh * D);
    load_row_f32<DV>(g, dO + (size_t)qh * DV);
    const float l = lse[qh];
    float p[NS], dp[NS], pv[NS];
    uint4 kw[kKeep ? NS : 1][D / 8];
    float dsum = 0.0f;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        p[s] = 0.0f;
        dp[s] = 0.0f;
        pv[s] = 0.0f;
        jj[s] = -1;
        const int slot = tl + 16 * s;
        // a pair exists wherever its index lies in [0, N), as the counting
        // pass sees it; its weight is zero if lse says no key was kept
        const int32_t j = slot < k ? idx[(size_t)qh * k + slot] : -1;
        if (j >= 0 && j < N) jj[s] = j;
        if (j >= 0 && j < N && l != -INFINITY) {
            {   // the key row (kept for dQ) and the two dot products
                uint4 w[D / 8];
                load_row_words<D>(w, K + ((size_t)j * H + h) * D);
                if constexpr (kKeep) {
#pragma unroll
                    for (int c = 0; c < D / 8; ++c) kw[s][c] = w[c];
                }
                const float z = scale * dot_words_bf16<D>(q, w);
                p[s] = __expf(z - l);
                dp[s] = dot_row_bf16<DV>(g, V + ((size_t)j * H + h) * DV);
                pv[s] = p[s];
                if (keep != nullptr) {
                    const float f = keep[(size_t)qh * k + slot] != 0 ? keep_scale : 0.0f;
                    dp[s] *= f;
                    pv[s] = p[s] * f;
                }
            }
        }
        dsum = fmaf(p[s], dp[s], dsum);
    }
    dsum = group16_sum(dsum);
    // dQ: each slot lane adds g_s k_j over its own slots, then the team
    // reduces the D-vector so that lane tl ends up with dimensions tl, tl+16, ...
    float acc[D];
#pragma unroll
    for (int t = 0; t < D; ++t) acc[t] = 0.0f;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        const float gs = p[s] * (dp[s] - dsum);
        ca[s] = scale * gs;
        cp[s] = pv[s];
        if (jj[s] >= 0 && l != -INFINITY) {
            uint4 w[D / 8];
            if constexpr (kKeep) {
#pragma unroll
                for (int c = 0; c < D / 8; ++c) w[c] = kw[s][c];
            } else {
                load_row_words<D>(w, K + ((size_t)jj[s] * H + h) * D);
            }
#pragma unroll
            for (int c = 0; c < D / 8; ++c) {
                const uint32_t ww[4] = {w[c].x, w[c].y, w[c].z, w[c].w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    acc[8 * c + 2 * e] = fmaf(gs, bf16_bits_to_f32(ww[e] & 0xFFFFu), acc[8 * c + 2 * e]);
                    acc[8 * c + 2 * e + 1] = fmaf(gs, bf16_bits_to_f32(ww[e] >> 16), acc[8 * c + 2 * e + 1]);
                }
            }
        }
    }
    float out[D / 16];
    team_sum_transpose<D>(acc, out, tl);
#pragma unroll
    for (int u = 0; u < D / 16; ++u) dQ[(size_t)qh * D + 16 * u + tl] = scale * out[u];
}

// The coefficients of every pair, in pair order (the segmented variant).
template <int D, int DV, int NS>
__global__ __launch_bounds__(256) void csr_coef_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K, const uint16_t* __restrict__ V,
    const uint16_t* __restrict__ dO, const int32_t* __restrict__ idx, const float* __restrict__ lse,
    int32_t N, int32_t H, int32_t k, float scale, float* __restrict__ dQ, float2* __restrict__ coef,
    uint16_t* __restrict__ QGt, const uint8_t* __restrict__ keep, float keep_scale) {
    const int tl = threadIdx.x & 15;
    const int64_t qh = (int64_t)blockIdx.x * 16 + (threadIdx.x >> 4);
    if (qh >= (int64_t)N * H) return;  // whole team exits together
    int32_t jj[NS];
    float ca[NS], cp[NS];
    coef_one<D, DV, NS>(Q, K, V, dO, idx, lse, keep, keep_scale, N, H, k, scale, qh, tl, dQ, QGt, 0, jj, ca, cp);
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        const int slot = tl + 16 * s;
        if (slot < k) coef[(size_t)qh * k + slot] = make_float2(ca[s], cp[s]);
    }
}

// Launches csr_coef_kernel<D, DV, NS> with NS the smallest power of two >= k/16.
template <int D, int DV>
void launch_coef(unsigned blocks, hipStream_t stream, const uint16_t* q, const uint16_t* kk,
                 const uint16_t* v, const uint16_t* g, const int32_t* idx, const float* lse, int32_t N,
                 int32_t H, int32_t k, float scale, float* dQ, float2* coef, uint16_t* qg, const uint8_t* keep,
                 float keep_scale) {
    const int ns = (k + 15) / 16;
    if (ns <= 1)
        hipLaunchKernelGGL((csr_coef_kernel<D, DV, 1>), dim3(blocks), dim3(256), 0, stream, q, kk, v, g, idx, lse,
                           N, H, k, scale, dQ, coef, qg, keep, keep_scale);
    else if (ns <= 2)
        hipLaunchKernelGGL((csr_coef_kernel<D, DV, 2>), dim3(blocks), dim3(256), 0, stream, q, kk, v, g, idx, lse,
                           N, H, k, scale, dQ, coef, qg, keep, keep_scale);
    else if (ns <= 4)
        hipLaunchKernelGGL((csr_coef_kernel<D, DV, 4>), dim3(blocks), dim3(256), 0, stream, q, kk, v, g, idx, lse,
                           N, H, k, scale, dQ, coef, qg, keep, keep_scale);
    else if (ns <= 8)
        hipLaunchKernelGGL((csr_coef_kernel<D, DV, 8>), dim3(blocks), dim3(256), 0, stream, q, kk, v, g, idx, lse,
                           N, H, k, scale, dQ, coef, qg, keep, keep_scale);
    else if constexpr (D <= 64) {
        // k > 128 (d <= 64 only)
        if (ns <= 16)
            hipLaunchKernelGGL((csr_coef_kernel<D, DV, 16>), dim3(blocks), dim3(256), 0, stream, q, kk, v, g, idx,
                               lse, N, H, k, scale, dQ, coef, qg, keep, keep_scale);
        else
            hipLaunchKernelGGL((csr_coef_kernel<D, DV, 32>), dim3(blocks), dim3(256), 0, stream, q, kk, v, g, idx,
                               lse, N, H, k, scale, dQ, coef, qg, keep, keep_scale);
    }
}

// Key row of slot s of query-head qh, or -1 (padding).
__device__ __forceinline__ int32_t pair_row(const int32_t* __restrict__ idx, int64_t qh, int s,
                                            int32_t k, int32_t N, int32_t H) {
    const int32_t j = idx[(size_t)qh * k + s];
    return (j >= 0 && j < N) ? j * H + (int32_t)(qh % H) : -1;
}

// 2 and 4.  A workgroup takes 256 query-heads (a thread each, walking its
// k slots) and first counts its pairs per key row in an LDS table, so that
// a key row most queries select costs one global atomic per workgroup.
// Rows that find no table slot count with their own global atomic.  The
// count pass adds the table's counts to cnt.  The place pass reserves a range
// of positions per table row with one atomic on the cursors (the scanned
// counts), then gives each pair the next position of its row's range and
// writes the pair's record there.
constexpr int kTab = 2048;      // table rows per workgroup
constexpr int kTabProbes = 8;

struct PairRecord {
    int32_t row;    // key row j*H + h
    int32_t qh;     // query-head i*H + h (full sort), or its head-major row h*N + i (buckets)
    float a;        // scale * g_ij
    float p;        // p_ij
};

struct CountTable {
    int32_t key[kTab];
    int32_t n[kTab];
    int32_t base[kTab];
};

// Slot of key row r in the table (claimed if absent), or -1 if every probe
// is taken by other rows.  With `claim` false, only looks up.
__device__ __forceinline__ int tab_slot(CountTable* t, int32_t r, bool claim) {
    const uint32_t hsh = ((uint32_t)r * 0x9E3779B1u) >> (32 - 11);
    for (int p = 0; p < kTabProbes; ++p) {
        const int ts = (int)((hsh + p) & (kTab - 1));
        const int32_t cur = __hip_atomic_load(&t->key[ts], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        if (cur == r) return ts;
        if (cur == -1) {
            if (!claim) return -1;
            const int32_t old = atomicCAS(&t->key[ts], -1, r);
            if (old == -1 || old == r) return ts;
        }
    }
    return -1;
}

template <bool kPlace>
__global__ __launch_bounds__(256) void csr_count_kernel(const int32_t* __restrict__ idx,
                                                        const float2* __restrict__ coef, int32_t N,
                                                        int32_t H, int32_t k,
                                                        int32_t* __restrict__ cnt,
                                                        PairRecord* __restrict__ rec) {
    static_assert(kTab == 1 << 11, "hash width");
    __shared__ CountTable tab;
    for (int e = threadIdx.x; e < kTab; e += 256) {
        tab.key[e] = -1;
        tab.n[e] = 0;
    }
    __syncthreads();
    const int64_t qh = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const bool live = qh < (int64_t)N * H;
    for (int s = 0; live && s < k; ++s) {
        const int32_t r = pair_row(idx, qh, s, k, N, H);
        if (r < 0) continue;
        const int ts = tab_slot(&tab, r, true);
        if (ts >= 0) {
            atomicAdd(&tab.n[ts], 1);
        } else if (kPlace) {
            const float2 c = coef[(size_t)qh * k + s];
            rec[atomicAdd(&cnt[r], 1)] = PairRecord{r, (int32_t)qh, c.x, c.y};
        } else {
            atomicAdd(&cnt[r], 1);
        }
    }
    __syncthreads();
    for (int e = threadIdx.x; e < kTab; e += 256) {
        const int32_t r = tab.key[e];
        if (r < 0 || tab.n[e] == 0) continue;
        const int32_t b = atomicAdd(&cnt[r], tab.n[e]);
        if (kPlace) tab.base[e] = b;
    }
    if constexpr (kPlace) {
        __syncthreads();
        for (int e = threadIdx.x; e < kTab; e += 256) tab.n[e] = 0;
        __syncthreads();
        for (int s = 0; live && s < k; ++s) {
            const int32_t r = pair_row(idx, qh, s, k, N, H);
            if (r < 0) continue;
            const int ts = tab_slot(&tab, r, false);
            if (ts < 0) continue;  // placed above
            const float2 c = coef[(size_t)qh * k + s];
            rec[tab.base[ts] + atomicAdd(&tab.n[ts], 1)] = PairRecord{r, (int32_t)qh, c.x, c.y};
        }
    }
}

// 3.  Exclusive scan of n counts in place: block sums, a scan of the block
// sums (one block), then each block's own scan plus its offset.
__device__ __forceinline__ int32_t block_exclusive_scan(int32_t v, int32_t* sh, int32_t* total) {
    const int t = threadIdx.x;
    sh[t] = v;
    __syncthreads();
    for (int off = 1; off < kScanBlock; off <<= 1) {
        const int32_t add = t >= off ? sh[t - off] : 0;
        __syncthreads();
        sh[t] += add;
        __syncthreads();
    }
    const int32_t incl = sh[t];
    if (total != nullptr && t == kScanBlock - 1) *total = incl;
    __syncthreads();
    return incl - v;
}

__global__ __launch_bounds__(kScanBlock) void scan_blocks_kernel(const int32_t* __restrict__ cnt,
                                                                 int64_t n, int32_t* __restrict__ sums) {
    __shared__ int32_t sh[kScanBlock];
    const int64_t i = (int64_t)blockIdx.x * kScanBlock + threadIdx.x;
    block_exclusive_scan(i < n ? cnt[i] : 0, sh, &sums[blockIdx.x]);
}

// Scans the nb block sums in place, kScanBlock at a time with a running
// carry; sums[nb] receives the grand total.
__global__ __launch_bounds__(kScanBlock) void scan_sums_kernel(int32_t* __restrict__ sums, int32_t nb) {
    __shared__ int32_t sh[kScanBlock];
    __shared__ int32_t total;
    const int t = threadIdx.x;
    int32_t carry = 0;
    for (int32_t base = 0; base < nb; base += kScanBlock) {
        const int32_t v = base + t < nb ? sums[base + t] : 0;
        const int32_t ex = block_exclusive_scan(v, sh, &total);
        if (base + t < nb) sums[base + t] = ex + carry;
        carry += total;
        __syncthreads();  // every thread has read total before it is rewritten
    }
    if (t == 0) sums[nb] = carry;
}

__global__ __launch_bounds__(kScanBlock) void scan_apply_kernel(int32_t* __restrict__ cnt, int64_t n,
                                                                const int32_t* __restrict__ sums) {
    __shared__ int32_t sh[kScanBlock];
    const int64_t i = (int64_t)blockIdx.x * kScanBlock + threadIdx.x;
    const int32_t ex = block_exclusive_scan(i < n ? cnt[i] : 0, sh, nullptr);
    if (i < n) cnt[i] = ex + sums[blockIdx.x];
}

// 5.  A wave per chunk of kChunk sorted pairs, four teams per wave, each team
// a contiguous quarter of the chunk.  `total` = number of sorted pairs.
template <int D, int DV>
__global__ __launch_bounds__(256) void csr_reduce_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ dO,
    const PairRecord* __restrict__ rec, const int32_t* __restrict__ total,
    float* __restrict__ dK, float* __restrict__ dV) {
    constexpr int U = D / 16;
    constexpr int UV = DV / 16;
    constexpr int kTeamSpan = kChunk / 4;
    const int tl = threadIdx.x & 15;
    const int team = (int)(blockIdx.x * 16 + (threadIdx.x >> 4));
    const int64_t e0 = (int64_t)team * kTeamSpan;
    const int64_t e1 = min((int64_t)*total, e0 + kTeamSpan);
    int32_t cur = -1;
    float ak[U], av[UV];
#pragma unroll
    for (int u = 0; u < U; ++u) ak[u] = 0.0f;
#pragma unroll
    for (int u = 0; u < UV; ++u) av[u] = 0.0f;
    auto flush = [&]() {
        if (cur >= 0) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                atomicAdd(dK + (size_t)cur * D + 16 * u + tl, ak[u]);
                ak[u] = 0.0f;
            }
#pragma unroll
            for (int u = 0; u < UV; ++u) {
                atomicAdd(dV + (size_t)cur * DV + 16 * u + tl, av[u]);
                av[u] = 0.0f;
            }
        }
    };
    for (int64_t b = e0; b < e1; b += 16) {
        // Sixteen records at a time: lane t fetches record b + t, then the
        // team walks them in order with each record broadcast.
        const int64_t e = b + tl;
        PairRecord r{-1, 0, 0.0f, 0.0f};
        if (e < e1) r = rec[e];
        const int n = (int)min((int64_t)16, e1 - b);
        for (int t = 0; t < n; ++t) {
            const int32_t rt = __shfl(r.row, t, 16);
            const int32_t qt = __shfl(r.qh, t, 16);
            const float at = __shfl(r.a, t, 16);
            const float pt = __shfl(r.p, t, 16);
            if (rt != cur) {
                flush();
                cur = rt;
            }
            const size_t qrow = (size_t)qt * D + tl;
            const size_t grow = (size_t)qt * DV + tl;
#pragma unroll
            for (int u = 0; u < U; ++u) ak[u] = fmaf(at, bf16_bits_to_f32(Q[qrow + 16 * u]), ak[u]);
#pragma unroll
            for (int u = 0; u < UV; ++u) av[u] = fmaf(pt, bf16_bits_to_f32(dO[grow + 16 * u]), av[u]);
        }
    }
    flush();
}

// ---- Variant 4: pairs bucketed by blocks of key rows, sorted in LDS ----
//
// The key rows are cut into buckets of RB consecutive rows, at most
// kMaxBuckets of them: RB = 4096 / d, doubled (up to kMaxBucketRows) while
// N*H would need more buckets.  The pairs are counting-sorted by bucket only: a
// counting pass takes ranges of consecutive pairs and counts them with an
// LDS histogram over the buckets, one global atomic per bucket it touches
// (against one per key row and workgroup for the full sort, whose per-row
// tables overflow when pairs spread over many keys); two placement passes
// (below) then write the records in bucket order.  Each bucket's records are
// cut into pieces that one workgroup sorts by key row in LDS and reduces
// like the full sort's reduction.
constexpr int kMaxBuckets = 8192;
constexpr int kMaxBucketRows = 512;

// log2 of the bucket rows for N*H key rows at width d (the bucketed variant
// takes N*H <= kMaxBuckets * kMaxBucketRows).
inline int bucket_shift(int64_t nh, int d) {
    int sh = d == 16 ? 8 : (d == 32 ? 7 : 6);
    while ((nh + (1 << sh) - 1) >> sh > kMaxBuckets && (1 << sh) < kMaxBucketRows) ++sh;
    return sh;
}

// Division of a dividend below 2^31 by a fixed divisor d >= 1 as a multiply
// and shift: with l = ceil(log2 d) and m = ceil(2^(32+l) / d) (at most 2^33),
// floor(n m / 2^(32+l)) = floor(n / d) for every n < 2^32 (the round-up
// method of Granlund and Montgomery); n < 2^31 keeps n m below 2^64.
struct FastDiv {
    uint64_t m;
    uint32_t s;
    uint32_t d;
};

inline FastDiv make_fastdiv(uint32_t d) {
    uint32_t l = 0;
    while ((1ull << l) < d) ++l;
    const unsigned __int128 num = (unsigned __int128)1 << (32 + l);
    return FastDiv{(uint64_t)((num + d - 1) / d), 32 + l, d};
}

__device__ __forceinline__ uint32_t fdiv(uint32_t n, const FastDiv& f) {
    return (uint32_t)(((uint64_t)n * f.m) >> f.s);
}

// A pair record of the bucketed sort, 12 bytes: the key row's offset in its
// bucket (below kMaxBucketRows = 2^9) in bits 22..30 and the head-major query
// row h*N + i in bits 0..21 (the bucketed variant takes N*H <= kMaxBuckets *
// kMaxBucketRows = 2^22), then the coefficients.
struct BucketRecord {
    uint32_t packed;
    float a;
    float p;
};
constexpr int kQRowBits = 22;
static_assert(sizeof(BucketRecord) == 12, "packed record");
static_assert((int64_t)kMaxBuckets * kMaxBucketRows <= (int64_t)1 << kQRowBits, "query rows fit 22 bits");
static_assert(kMaxBucketRows <= 1 << (32 - kQRowBits), "bucket offsets fit the other 10 bits");

// Takes one slot of LDS counter ctr[bk] for each lane with bk >= 0 and
// returns its number (kReturn) or nothing.  Lanes of a wave that share a bucket are served
// by one atomic while the group the wave's first pending lane belongs to
// holds at least 8 lanes (a bucket most pairs fall in: one atomic per wave
// instead of one per lane); the rest take one atomic each.
template <bool kReturn>
__device__ __forceinline__ int32_t claim_slot(int32_t* ctr, int32_t bk) {
    const int lane = threadIdx.x & 63;
    bool pending = bk >= 0;
    int32_t slot = 0;
    for (int it = 0; it < 4; ++it) {
        const uint64_t act = __ballot(pending);
        if (act == 0) break;
        int32_t grp = 0;
        if (pending) {
            const int32_t b0 = __builtin_amdgcn_readfirstlane(bk);
            const uint64_t eq = __ballot(bk == b0);
            grp = __popcll(eq);
            if (grp >= 8) {
                const int leader = __ffsll((unsigned long long)eq) - 1;
                int32_t base0 = 0;
                if (lane == leader) base0 = atomicAdd(&ctr[b0], grp);
                if (kReturn) base0 = __shfl(base0, leader, 64);
                if (bk == b0) {
                    slot = base0 + (int32_t)__popcll(eq & ((1ull << lane) - 1ull));
                    pending = false;
                }
            }
        }
        // this round's group size, as seen by its first lane
        if (__builtin_amdgcn_readlane(grp, __ffsll((unsigned long long)act) - 1) < 8) break;
    }
    if (pending) slot = atomicAdd(&ctr[bk], 1);
    return slot;
}

// Counting pass over a range of `per` consecutive pairs (pair e =
// query-head e / k, slot e % k, so that lanes read idx contiguously): the
// workgroup counts its pairs per bucket in LDS and adds the counts to the
// global ones, one atomic per bucket it touches.
__global__ __launch_bounds__(256) void bkt_count_kernel(const int32_t* __restrict__ idx, int32_t N, int32_t H,
                                                        int32_t k, FastDiv divk, FastDiv divh, int32_t shift,
                                                        int32_t nbk, uint32_t per, int32_t* __restrict__ gcnt) {
    __shared__ int32_t hist[kMaxBuckets];
    const int t = threadIdx.x;
    const uint32_t P = (uint32_t)N * (uint32_t)H * (uint32_t)k;
    const uint32_t p0 = blockIdx.x * per;
    const uint32_t p1 = min(P, p0 + per);
    auto row_of = [&](uint32_t e) -> int32_t {
        if (e >= p1) return -1;
        const int32_t j = idx[e];
        const uint32_t qh = fdiv(e, divk);
        return (j >= 0 && j < N) ? j * H + (int32_t)(qh - fdiv(qh, divh) * (uint32_t)H) : -1;
    };
    for (int e = t; e < nbk; e += 256) hist[e] = 0;
    __syncthreads();
    // every lane runs the same number of rounds (wave-wide claims); four
    // pairs' loads are issued before their claims
    for (uint32_t pb = p0; pb < p1; pb += 1024) {
        int32_t r[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) r[u] = row_of(pb + 256 * u + t);
#pragma unroll
        for (int u = 0; u < 4; ++u) claim_slot<false>(hist, r[u] >= 0 ? r[u] >> shift : -1);
    }
    __syncthreads();
    for (int e = t; e < nbk; e += 256) {
        const int32_t c = hist[e];
        if (c != 0) atomicAdd(&gcnt[e], c);
    }
}


// Placing the records in bucket order takes two passes with coalesced
// stores (a single pass that sends each pair to its bucket directly makes
// one scattered store per pair).  Pass 1, fused with the coefficient pass
// (coef_split_kernel), sorts each chunk of kSplitChunk pairs by super-bucket
// (kSupBuckets consecutive buckets, at most kMaxBuckets / kSupBuckets of
// them) in LDS, reserves each super-bucket's range with one atomic and
// writes the chunk out as runs; pass 2 does the same for each piece of
// kSplitChunk records of one super-bucket, by bucket, and writes the final
// records.
constexpr int kSplitChunk = 2048;
constexpr int kSupBuckets = 128;
constexpr int kMaxSup = kMaxBuckets / kSupBuckets;
static_assert(kMaxSup == 64 && kSupBuckets == 128, "6-bit super-bucket and 7-bit bucket digits; one-wave scans");

// Exclusive prefix sum over the 64 lanes of a wave; *total (lane 63's
// inclusive sum) for every lane.
__device__ __forceinline__ int32_t wave_exclusive_sum(int32_t v, int32_t* total) {
    const int lane = threadIdx.x & 63;
    int32_t x = v;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int32_t y = __shfl_up(x, off, 64);
        if (lane >= off) x += y;
    }
    *total = __shfl(x, 63, 64);
    return x - v;
}

// Slot of each lane with digit >= 0 (a value below 2^NB) in LDS counter
// ctr[digit]: the lanes of the wave with equal digits are found with NB
// ballots, and one leader per digit takes the group's slots with a single
// atomic (lanes with equal digits never meet at one counter in an atomic).
template <int NB>
__device__ __forceinline__ int32_t wave_rank(int32_t* ctr, int32_t digit) {
    const int lane = threadIdx.x & 63;
    uint64_t same = __ballot(digit >= 0);
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        const bool bit = ((digit >> b) & 1) != 0;
        const uint64_t bb = __ballot(bit);
        same &= bit ? bb : ~bb;
    }
    const int leader = same != 0ull ? __ffsll((unsigned long long)same) - 1 : lane;
    int32_t base = 0;
    if (digit >= 0 && lane == leader) base = atomicAdd(&ctr[digit], (int32_t)__popcll(same));
    base = __shfl(base, leader, 64);
    return base + (int32_t)__popcll(same & ((1ull << lane) - 1ull));
}

// Inputs of one query-head of the coefficient pass, fetched one query-head
// ahead (coef_fetch) so that their loads overlap the previous query-head's
// arithmetic (coef_compute).
template <int D, int NS>
struct CoefIn {
    int32_t j[NS];       // this lane's key slots tl + 16 s (-1: none)
    uint4 qw[D / 8];     // q_i and dO_i as bf16 words
    uint4 gw[D / 8];
    float l;             // lse (-inf: no key kept, or no query-head)
    int64_t qh;
    bool valid;          // u < N H
};

template <int D, int NS>
__device__ __forceinline__ void coef_fetch(const uint16_t* __restrict__ Q, const uint16_t* __restrict__ dO,
                                           const int32_t* __restrict__ idx, const float* __restrict__ lse,
                                           int32_t N, int32_t H, int32_t k, int64_t u, int64_t nh, int32_t i, int tl,
                                           CoefIn<D, NS>& in) {
    in.valid = u < nh;
    const int32_t h = in.valid ? (int32_t)(u / N) : 0;
    in.qh = (int64_t)i * H + h;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        const int slot = tl + 16 * s;
        in.j[s] = in.valid && slot < k ? idx[(size_t)in.qh * k + slot] : -1;
    }
    if (in.valid) {
        load_row_words<D>(in.qw, Q + (size_t)in.qh * D);
        load_row_words<D>(in.gw, dO + (size_t)in.qh * D);
        in.l = lse[in.qh];
    } else {
#pragma unroll
        for (int c = 0; c < D / 8; ++c) in.qw[c] = in.gw[c] = make_uint4(0, 0, 0, 0);
        in.l = -INFINITY;
    }
}

// coef_one's arithmetic (value width D, with the interleaved copy) on
// fetched inputs: the same operations in the same order, so the same bits.
// (A coef_one built from coef_fetch and coef_compute, which would leave one
// copy of the arithmetic, made the code the compiler emits for width 32
// slower: the backward went from 1.10 to 1.39 ms on a 100k-node
// graph at d = 32, so the two stay apart.)
template <int D, int NS>
__device__ __forceinline__ void coef_compute(const CoefIn<D, NS>& in, const uint16_t* __restrict__ K,
                                             const uint16_t* __restrict__ V, const uint8_t* __restrict__ keep,
                                             float keep_scale, int32_t N, int32_t H, int32_t k, float scale,
                                             int tl, float* __restrict__ dQ, uint16_t* __restrict__ QGt,
                                             size_t qg_row, int32_t (&jj)[NS], float (&ca)[NS], float (&cp)[NS]) {
    constexpr bool kKeep = D / 2 * NS <= 64;
    const int64_t qh = in.qh;
    const int h = (int)(qh % H);
    if (in.valid && tl < D / 4) {
        // row qg_row of the interleaved copy: lane tl < D / 8 writes chunk tl
        // of q_i, lane D / 8 + c chunk c of dO_i
        uint4 v = in.qw[0];
#pragma unroll
        for (int c = 1; c < D / 8; ++c)
            if (tl == c) v = in.qw[c];
#pragma unroll
        for (int c = 0; c < D / 8; ++c)
            if (tl == D / 8 + c) v = in.gw[c];
        reinterpret_cast<uint4*>(QGt + qg_row * (2 * D))[tl] = v;
    }
    float q[D], g[D];
#pragma unroll
    for (int c = 0; c < D / 8; ++c) {
        const uint32_t wq[4] = {in.qw[c].x, in.qw[c].y, in.qw[c].z, in.qw[c].w};
        const uint32_t wg[4] = {in.gw[c].x, in.gw[c].y, in.gw[c].z, in.gw[c].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            q[8 * c + 2 * e] = bf16_bits_to_f32(wq[e] & 0xFFFFu);
            q[8 * c + 2 * e + 1] = bf16_bits_to_f32(wq[e] >> 16);
            g[8 * c + 2 * e] = bf16_bits_to_f32(wg[e] & 0xFFFFu);
            g[8 * c + 2 * e + 1] = bf16_bits_to_f32(wg[e] >> 16);
        }
    }
    const float l = in.l;
    float p[NS], dp[NS], pv[NS];
    uint4 kw[kKeep ? NS : 1][D / 8];
    float dsum = 0.0f;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        p[s] = 0.0f;
        dp[s] = 0.0f;
        pv[s] = 0.0f;
        jj[s] = -1;
        const int slot = tl + 16 * s;
        const int32_t j = in.j[s];
        if (j >= 0 && j < N) jj[s] = j;
        if (j >= 0 && j < N && l != -INFINITY) {
            uint4 w[D / 8];
            load_row_words<D>(w, K + ((size_t)j * H + h) * D);
            if constexpr (kKeep) {
#pragma unroll
                for (int c = 0; c < D / 8; ++c) kw[s][c] = w[c];
            }
            const float z = scale * dot_words_bf16<D>(q, w);
            p[s] = __expf(z - l);
            dp[s] = dot_row_bf16<D>(g, V + ((size_t)j * H + h) * D);
            pv[s] = p[s];
            if (keep != nullptr) {
                const float f = keep[(size_t)qh * k + slot] != 0 ? keep_scale : 0.0f;
                dp[s] *= f;
                pv[s] = p[s] * f;
            }
        }
        dsum = fmaf(p[s], dp[s], dsum);
    }
    dsum = group16_sum(dsum);
    float acc[D];
#pragma unroll
    for (int t = 0; t < D; ++t) acc[t] = 0.0f;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        const float gs = p[s] * (dp[s] - dsum);
        ca[s] = scale * gs;
        cp[s] = pv[s];
        if (jj[s] >= 0 && l != -INFINITY) {
            uint4 w[D / 8];
            if constexpr (kKeep) {
#pragma unroll
                for (int c = 0; c < D / 8; ++c) w[c] = kw[s][c];
            } else {
                load_row_words<D>(w, K + ((size_t)jj[s] * H + h) * D);
            }
#pragma unroll
            for (int c = 0; c < D / 8; ++c) {
                const uint32_t ww[4] = {w[c].x, w[c].y, w[c].z, w[c].w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    acc[8 * c + 2 * e] = fmaf(gs, bf16_bits_to_f32(ww[e] & 0xFFFFu), acc[8 * c + 2 * e]);
                    acc[8 * c + 2 * e + 1] = fmaf(gs, bf16_bits_to_f32(ww[e] >> 16), acc[8 * c + 2 * e + 1]);
                }
            }
        }
    }
    float out[D / 16];
    team_sum_transpose<D>(acc, out, tl);
    if (in.valid) {
#pragma unroll
        for (int u = 0; u < D / 16; ++u) dQ[(size_t)qh * D + 16 * u + tl] = scale * out[u];
    }
}

// The coefficient pass fused with placement pass 1: a
// workgroup takes 128 / NS query-heads (8 / NS per team, at most 2048
// pairs), computes their coefficients, dQ and the interleaved copy, and
// writes their records in super-bucket order: one record per lane and
// round for 8 rounds, ranked by ballots, staged in LDS and written as runs
// into ranges the workgroup reserves with one atomic per super-bucket.  The
// coefficients never go to memory.
// The query-heads are taken in the order u = h N + p, query perm[h][p] at
// position p of head h: with perm the grouping of the queries by direction,
// queries that share most of their keys are processed together (their key
// and value rows are gathered while in cache) and their rows of the
// interleaved copy, row u, lie side by side, so the reduction's gathers for
// one key row mostly read neighbouring rows and share cache lines.  The
// records carry u as their query row.
template <int D, int NS>
__global__ __launch_bounds__(256) void coef_split_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K, const uint16_t* __restrict__ V,
    const uint16_t* __restrict__ dO, const int32_t* __restrict__ idx, const float* __restrict__ lse,
    const int32_t* __restrict__ perm, int32_t N, int32_t H, int32_t k, float scale, float* __restrict__ dQ,
    uint16_t* __restrict__ QGt, int32_t shift, int32_t* __restrict__ supcur, PairRecord* __restrict__ mid,
    const uint8_t* __restrict__ keep, float keep_scale) {
    constexpr int TQ = 8 / NS;   // query-heads per team
    constexpr int R = TQ * NS;   // records per lane: 8
    static_assert(256 * R == kSplitChunk, "one staging chunk per workgroup");
    __shared__ int32_t cnt[kMaxSup], lstart[kMaxSup], gbase[kMaxSup];
    __shared__ PairRecord stage[kSplitChunk];
    __shared__ int32_t total;
    const int t = threadIdx.x;
    const int tl = t & 15, team = t >> 4;
    const int64_t nh = (int64_t)N * H;
    if (t < kMaxSup) cnt[t] = 0;
    PairRecord rr[R];
    int32_t sup[R], slot[R];
    // With narrow rows the inputs of a team's next query-head are fetched
    // while the current one computes (the query rows of all of them first);
    // wider rows would not leave the registers for it.
    constexpr bool kAhead = D == 16 || (D == 32 && NS == 1);
    int32_t qrow[TQ];
    CoefIn<D, NS> nxt;
    if constexpr (kAhead) {
#pragma unroll
        for (int it = 0; it < TQ; ++it) {
            const int64_t u = (int64_t)blockIdx.x * (16 * TQ) + it * 16 + team;
            qrow[it] = u < nh ? perm[u] : 0;
        }
        coef_fetch<D, NS>(Q, dO, idx, lse, N, H, k, (int64_t)blockIdx.x * (16 * TQ) + team, nh, qrow[0], tl, nxt);
    }
#pragma unroll
    for (int it = 0; it < TQ; ++it) {
        const int64_t u = (int64_t)blockIdx.x * (16 * TQ) + it * 16 + team;
        const int32_t h = u < nh ? (int32_t)(u / N) : 0;
        int32_t jj[NS];
        float ca[NS], cp[NS];
        if constexpr (kAhead) {
            const CoefIn<D, NS> cur = nxt;
            if (it + 1 < TQ)
                coef_fetch<D, NS>(Q, dO, idx, lse, N, H, k, u + 16, nh, qrow[it + 1], tl, nxt);
            coef_compute<D, NS>(cur, K, V, keep, keep_scale, N, H, k, scale, tl, dQ, QGt, (size_t)u, jj, ca, cp);
        } else {
            const int32_t i = u < nh ? perm[u] : 0;
            const int64_t qh = (int64_t)i * H + h;
#pragma unroll
            for (int s2 = 0; s2 < NS; ++s2) jj[s2] = -1;
            if (u < nh)
                coef_one<D, D, NS>(Q, K, V, dO, idx, lse, keep, keep_scale, N, H, k, scale, qh, tl, dQ, QGt,
                                   (size_t)u, jj, ca, cp);
        }
#pragma unroll
        for (int s2 = 0; s2 < NS; ++s2) {
            const int r = it * NS + s2;
            sup[r] = -1;
            rr[r] = PairRecord{-1, 0, 0.0f, 0.0f};
            if (u < nh && jj[s2] >= 0) {
                const int32_t row = jj[s2] * H + h;
                rr[r] = PairRecord{row, (int32_t)u, ca[s2], cp[s2]};
                sup[r] = (row >> shift) / kSupBuckets;
            }
        }
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < R; ++r) slot[r] = wave_rank<6>(cnt, sup[r]);
    __syncthreads();
    if (t < 64) {
        const int32_t c = t < kMaxSup ? cnt[t] : 0;
        int32_t tot;
        const int32_t ex = wave_exclusive_sum(c, &tot);
        if (t < kMaxSup) {
            lstart[t] = ex;
            gbase[t] = c != 0 ? atomicAdd(&supcur[t], c) : 0;
        }
        if (t == 0) total = tot;
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < R; ++r)
        if (sup[r] >= 0) stage[lstart[sup[r]] + slot[r]] = rr[r];
    __syncthreads();
    const int n = total;
    for (int j = t; j < n; j += 256) {
        const PairRecord rec = stage[j];
        const int sp = (rec.row >> shift) / kSupBuckets;
        mid[gbase[sp] + (j - lstart[sp])] = rec;
    }
}

template <int D>
hipError_t launch_coef_split(int32_t nh, hipStream_t stream, const uint16_t* q, const uint16_t* kk,
                             const uint16_t* v, const uint16_t* g, const int32_t* idx, const float* lse,
                             const int32_t* perm, int32_t N, int32_t H, int32_t k, float scale, float* dQ,
                             uint16_t* qg, int32_t shift, int32_t* supcur, PairRecord* mid, const uint8_t* keep,
                             float keep_scale) {
    const int ns = (k + 15) / 16;
#define KMIP_COEF_SPLIT(NSV)                                                                           \
    hipLaunchKernelGGL((coef_split_kernel<D, NSV>), dim3((unsigned)((nh + 128 / NSV - 1) / (128 / NSV))),   \
                       dim3(256), 0, stream, q, kk, v, g, idx, lse, perm, N, H, k, scale, dQ, qg, shift, supcur, mid, \
                       keep, keep_scale)
    if (ns <= 1)
        KMIP_COEF_SPLIT(1);
    else if (ns <= 2)
        KMIP_COEF_SPLIT(2);
    else if (ns <= 4)
        KMIP_COEF_SPLIT(4);
    else
        KMIP_COEF_SPLIT(8);
#undef KMIP_COEF_SPLIT
    return hipGetLastError();
}

// Per super-bucket: its first record (supst, nsup + 1 entries), the cursor
// pass 1 reserves from (supcur), and the scanned number of pass-2 pieces
// (pstart2, nsup + 1 entries).  One wave.
__global__ __launch_bounds__(64) void bkt_split_setup_kernel(const int32_t* __restrict__ sstart, int32_t nbk,
                                                             int32_t nsup, int32_t* __restrict__ supst,
                                                             int32_t* __restrict__ supcur,
                                                             int32_t* __restrict__ pstart2) {
    const int s = threadIdx.x;
    const int32_t a = sstart[min(s * kSupBuckets, nbk)];
    const int32_t b = sstart[min((s + 1) * kSupBuckets, nbk)];
    const int32_t np = s < nsup ? (b - a + kSplitChunk - 1) / kSplitChunk : 0;
    int32_t tot;
    const int32_t ex = wave_exclusive_sum(np, &tot);
    if (s < nsup) {
        supst[s] = a;
        supcur[s] = a;
        pstart2[s] = ex;
    }
    if (s == 0) {
        supst[nsup] = sstart[nbk];
        pstart2[nsup] = tot;
    }
}

// Pass 2: one workgroup per piece of at most kSplitChunk records of one
// super-bucket; bcur holds the buckets' cursors (their starts, advanced
// here).
__global__ __launch_bounds__(256) void bkt_split2_kernel(const PairRecord* __restrict__ mid,
                                                         const int32_t* __restrict__ supst,
                                                         const int32_t* __restrict__ pstart2, int32_t nsup,
                                                         int32_t shift, int32_t* __restrict__ bcur,
                                                         BucketRecord* __restrict__ rec) {
    constexpr int R = kSplitChunk / 256;
    __shared__ int32_t cnt[kSupBuckets], lstart[kSupBuckets], gbase[kSupBuckets];
    __shared__ BucketRecord stage[kSplitChunk];
    __shared__ uint8_t sbk[kSplitChunk];
    const int t = threadIdx.x;
    const int w = blockIdx.x;
    if (w >= pstart2[nsup]) return;
    int lo = 0, hi = nsup;
    while (hi - lo > 1) {
        const int m = (lo + hi) >> 1;
        if (pstart2[m] <= w) lo = m; else hi = m;
    }
    const int32_t e0 = supst[lo] + (w - pstart2[lo]) * kSplitChunk;
    const int32_t n = min(supst[lo + 1] - e0, kSplitChunk);
    const int32_t b0 = lo * kSupBuckets;
    if (t < kSupBuckets) cnt[t] = 0;
    __syncthreads();
    BucketRecord fr[R];
    int32_t bk[R], slot[R];
    const uint32_t offmask = (1u << shift) - 1u;
#pragma unroll
    for (int u = 0; u < R; ++u) {
        const int i = u * 256 + t;
        bk[u] = -1;
        fr[u] = BucketRecord{0u, 0.0f, 0.0f};
        if (i < n) {
            const PairRecord r = mid[e0 + i];
            bk[u] = (r.row >> shift) - b0;
            fr[u] = BucketRecord{(((uint32_t)r.row & offmask) << kQRowBits) | (uint32_t)r.qh, r.a, r.p};
        }
    }
#pragma unroll
    for (int u = 0; u < R; ++u) slot[u] = wave_rank<7>(cnt, bk[u]);
    __syncthreads();
    if (t < 64) {
        // two halves of kSupBuckets = 128 counters, one wave
        const int32_t c0 = cnt[t], c1 = cnt[t + 64];
        int32_t tot0, tot1;
        const int32_t ex0 = wave_exclusive_sum(c0, &tot0);
        const int32_t ex1 = wave_exclusive_sum(c1, &tot1);
        lstart[t] = ex0;
        lstart[t + 64] = tot0 + ex1;
        gbase[t] = c0 != 0 ? atomicAdd(&bcur[b0 + t], c0) : 0;
        gbase[t + 64] = c1 != 0 ? atomicAdd(&bcur[b0 + t + 64], c1) : 0;
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < R; ++u) {
        if (bk[u] >= 0) {
            stage[lstart[bk[u]] + slot[u]] = fr[u];
            sbk[lstart[bk[u]] + slot[u]] = (uint8_t)bk[u];
        }
    }
    __syncthreads();
    for (int i = t; i < n; i += 256) {
        const int b = sbk[i];
        rec[gbase[b] + (i - lstart[b])] = stage[i];
    }
}

constexpr int kPiece = 8192;   // records per reduction workgroup (fits a uint16 order)

// After the scan: the start of each bucket's records (kept; the place pass
// moves the cursors) and its number of pieces of at most kPiece records.
__global__ __launch_bounds__(256) void bkt_pieces_kernel(const int32_t* __restrict__ start, int32_t nbk,
                                                         int32_t* __restrict__ sstart,
                                                         int32_t* __restrict__ npieces) {
    const int b = blockIdx.x * 256 + threadIdx.x;
    if (b > nbk) return;
    sstart[b] = start[b];
    if (b < nbk) npieces[b] = (start[b + 1] - start[b] + kPiece - 1) / kPiece;
    else npieces[b] = 0;
}

// One workgroup per piece (a stretch of at most kPiece records of one
// bucket, found by binary search in the scanned piece counts):
//   1. counting sort of the piece's records by key row in LDS (claim_slot:
//      a key most pairs share costs about one LDS atomic per wave);
//   2. sixteen teams of 16 lanes walk contiguous stretches of the sorted
//      order.  A record's query row of the interleaved head-major copy
//      (q then dO, 4d bytes) is one load per team, lane tl taking d/8
//      elements: lanes 0-7 hold q and add a*q to dK, lanes 8-15 hold dO and
//      add p*dO to dV.  Head-major rows let a key's run of queries of one
//      head read consecutive rows.  A team keeps the sums of the current key
//      row in registers and adds them to dK and dV (zero at the start) with
//      one atomic per dimension where the row changes or the stretch ends; it
//      loads the rows of eight pairs before adding them up.
template <int E>
struct RowChunk;   // E bf16 values, one load
template <> struct RowChunk<2> { uint32_t w[1]; };
template <> struct RowChunk<4> { uint32_t w[2]; };
template <> struct RowChunk<8> { uint32_t w[4]; };

template <int E>
__device__ __forceinline__ RowChunk<E> load_chunk(const uint16_t* p) {
    RowChunk<E> c;
    if constexpr (E == 2) {
        c.w[0] = *reinterpret_cast<const uint32_t*>(p);
    } else if constexpr (E == 4) {
        const uint2 v = *reinterpret_cast<const uint2*>(p);
        c.w[0] = v.x;
        c.w[1] = v.y;
    } else {
        const uint4 v = *reinterpret_cast<const uint4*>(p);
        c.w[0] = v.x;
        c.w[1] = v.y;
        c.w[2] = v.z;
        c.w[3] = v.w;
    }
    return c;
}

template <int D, int RB>
__global__ __launch_bounds__(256) void bkt_reduce_kernel(const uint16_t* __restrict__ QG,
                                                         const BucketRecord* __restrict__ rec,
                                                         const int32_t* __restrict__ sstart,
                                                         const int32_t* __restrict__ pstart, int32_t nbk,
                                                         float* __restrict__ dK, float* __restrict__ dV) {
    constexpr int E = D / 8;            // elements of the interleaved row per lane
    constexpr int G = 8;                // pairs whose rows a team loads at once
    constexpr int CPT = (RB + 255) / 256;   // cursors per thread in the scan
    using LRow = typename std::conditional<(RB <= 256), uint8_t, uint16_t>::type;
    __shared__ uint16_t ord[kPiece];
    __shared__ LRow lrow[kPiece];
    __shared__ int32_t cursor[RB];
    __shared__ int32_t sh[256];
    const int t = threadIdx.x;
    const int w = blockIdx.x;
    if (w >= pstart[nbk]) return;
    // bucket b with pstart[b] <= w < pstart[b + 1]
    int lo = 0, hi = nbk;
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (pstart[mid] <= w) lo = mid; else hi = mid;
    }
    const int32_t e0 = sstart[lo] + (w - pstart[lo]) * kPiece;
    const int32_t n = min(sstart[lo + 1] - e0, kPiece);
    for (int r = t; r < RB; r += 256) cursor[r] = 0;
    __syncthreads();

    // 1a. records per key row; the rows (local to the bucket) are kept in LDS
    for (int base = 0; base < n; base += 1024) {
        int32_t row[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int i = base + 256 * u + t;
            row[u] = i < n ? (int32_t)(rec[e0 + i].packed >> kQRowBits) : -1;
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int i = base + 256 * u + t;
            if (row[u] >= 0) lrow[i] = (LRow)row[u];
            claim_slot<false>(cursor, row[u]);
        }
    }
    __syncthreads();
    // 1b. exclusive scan of the counts: the cursors (thread t owns cursors
    // CPT t .. CPT t + CPT - 1)
    int32_t c = 0;
#pragma unroll
    for (int j = 0; j < CPT; ++j) c += CPT * t + j < RB ? cursor[CPT * t + j] : 0;
    sh[t] = c;
    __syncthreads();
    for (int off = 1; off < 256; off <<= 1) {
        const int32_t add = t >= off ? sh[t - off] : 0;
        __syncthreads();
        sh[t] += add;
        __syncthreads();
    }
    int32_t run = sh[t] - c;
#pragma unroll
    for (int j = 0; j < CPT; ++j) {
        if (CPT * t + j < RB) {
            const int32_t v = cursor[CPT * t + j];
            cursor[CPT * t + j] = run;
            run += v;
        }
    }
    __syncthreads();
    // 1c. place the record numbers in key-row order
    for (int base = 0; base < n; base += 256) {
        const int i = base + t;
        const int32_t row = i < n ? (int32_t)lrow[i] : -1;
        const int32_t slot = claim_slot<true>(cursor, row);
        if (row >= 0) ord[slot] = (uint16_t)i;
    }
    __syncthreads();

    // 2. teams walk the sorted order
    const int tl = t & 15;
    const int team = t >> 4;
    const bool isq = tl < 8;
    const int span = (n + 15) / 16;
    const int p0 = min(n, team * span), p1 = min(n, p0 + span);
    int32_t cur = -1;
    float acc[E];
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] = 0.0f;
    float* const dst0 = (isq ? dK : dV) + (tl & 7) * E;
    auto flush = [&]() {
        if (cur >= 0) {
#pragma unroll
            for (int e = 0; e < E; ++e) {
                atomicAdd(dst0 + (size_t)cur * D + e, acc[e]);
                acc[e] = 0.0f;
            }
        }
    };
    const int32_t row0 = lo * RB;   // first key row of the bucket
    BucketRecord next{0u, 0.0f, 0.0f};
    if (p0 + tl < p1) next = rec[e0 + ord[p0 + tl]];
    for (int pb = p0; pb < p1; pb += 16) {
        const BucketRecord r = next;   // this batch's records; the next batch's are fetched now
        next = BucketRecord{0u, 0.0f, 0.0f};
        if (pb + 16 + tl < p1) next = rec[e0 + ord[pb + 16 + tl]];
        const int m = min(16, p1 - pb);
        for (int s0 = 0; s0 < m; s0 += G) {
            int32_t rt[G];
            float ct[G];
            RowChunk<E> rv[G];
#pragma unroll
            for (int g = 0; g < G; ++g) {
                const uint32_t pk = (uint32_t)__shfl((int32_t)r.packed, s0 + g, 16);
                rt[g] = row0 + (int32_t)(pk >> kQRowBits);
                const int32_t qt = (int32_t)(pk & ((1u << kQRowBits) - 1u));
                // lanes 0-7 take the record's a, lanes 8-15 its p
                const float ca = __shfl(r.a, s0 + g, 16), cp = __shfl(r.p, s0 + g, 16);
                ct[g] = isq ? ca : cp;
                if (s0 + g < m) {
                    rv[g] = load_chunk<E>(QG + (size_t)qt * (2 * D) + tl * E);
                } else {
#pragma unroll
                    for (int w = 0; w < E / 2; ++w) rv[g].w[w] = 0u;
                }
            }
#pragma unroll
            for (int g = 0; g < G; ++g) {
                if (s0 + g >= m) break;
                if (rt[g] != cur) {
                    flush();
                    cur = rt[g];
                }
#pragma unroll
                for (int w = 0; w < E / 2; ++w) {
                    acc[2 * w] = fmaf(ct[g], bf16_bits_to_f32(rv[g].w[w] & 0xFFFFu), acc[2 * w]);
                    acc[2 * w + 1] = fmaf(ct[g], bf16_bits_to_f32(rv[g].w[w] >> 16), acc[2 * w + 1]);
                }
            }
        }
    }
    flush();
}

// perm[h][p] = p: the plain query order, in the layout of a grouping.
__global__ __launch_bounds__(256) void identity_order_kernel(int32_t N, int32_t H, int32_t* __restrict__ perm) {
    const int64_t u = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (u < (int64_t)N * H) perm[u] = (int32_t)(u % N);
}

}  // namespace

bool bwd_bucket_supported(int32_t N, int32_t H, int32_t d, int32_t k) {
    // the coefficient pass is built for d <= 64 and at most 8 slots a lane
    if (d > 64 || k > 128) return false;
    const int64_t nh = (int64_t)N * H;
    const int sh = bucket_shift(nh, d);
    return ((nh + (1 << sh) - 1) >> sh) <= kMaxBuckets;
}

size_t bwd_bucket_workspace_bytes(int32_t N, int32_t H, int32_t d, int32_t k) {
    auto al = [](size_t x) { return (x + 255) / 256 * 256; };
    const size_t nh = (size_t)N * H, pairs = nh * k;
    const size_t nbk = (nh + ((size_t)1 << bucket_shift((int64_t)nh, d)) - 1) >> bucket_shift((int64_t)nh, d);
    const size_t nb = (nbk + 1 + kScanBlock - 1) / kScanBlock;
    return al(pairs * sizeof(BucketRecord)) + 3 * al((nbk + 1) * sizeof(int32_t)) +
           al((nb + 1) * sizeof(int32_t)) + al(nh * 2 * d * sizeof(uint16_t)) + al(pairs * sizeof(PairRecord)) +
           3 * al((kMaxSup + 1) * sizeof(int32_t)) + al(group_workspace_bytes(N, H, d));
}

hipError_t launch_bwd_bucket(const void* Q, const void* K, const void* V, const void* dO,
                             const int32_t* idx, const float* lse, const uint8_t* keep, float keep_scale,
                             int32_t N, int32_t H, int32_t d, int32_t k, float scale, float* dQ, float* dK,
                             float* dV, void* ws, hipStream_t stream) {
    auto al = [](size_t x) { return (x + 255) / 256 * 256; };
    const int64_t nh = (int64_t)N * H;
    if (nh == 0) return hipSuccess;
    const size_t pairs = (size_t)nh * k;
    const int32_t shift = bucket_shift(nh, d);
    const int32_t rb = 1 << shift;
    const int32_t nbk = (int32_t)((nh + rb - 1) / rb);
    if (nbk > kMaxBuckets) return hipErrorInvalidValue;
    const int32_t nb = (nbk + 1 + kScanBlock - 1) / kScanBlock;
    char* p = reinterpret_cast<char*>(ws);
    BucketRecord* rec = reinterpret_cast<BucketRecord*>(p);
    p += al(pairs * sizeof(BucketRecord));
    int32_t* gcnt = reinterpret_cast<int32_t*>(p);   // counts, then starts (nbk + 1 entries)
    p += al(((size_t)nbk + 1) * sizeof(int32_t));
    int32_t* sstart = reinterpret_cast<int32_t*>(p);   // kept starts
    p += al(((size_t)nbk + 1) * sizeof(int32_t));
    int32_t* pstart = reinterpret_cast<int32_t*>(p);   // pieces per bucket, then their starts
    p += al(((size_t)nbk + 1) * sizeof(int32_t));
    int32_t* sums = reinterpret_cast<int32_t*>(p);
    p += al(((size_t)nb + 1) * sizeof(int32_t));
    uint16_t* qg = reinterpret_cast<uint16_t*>(p);   // q and dO interleaved, row h N + p for query perm[h][p]
    p += al((size_t)nh * 2 * d * sizeof(uint16_t));
    PairRecord* mid = reinterpret_cast<PairRecord*>(p);   // records in super-bucket order (pass 1)
    p += al(pairs * sizeof(PairRecord));
    int32_t* supst = reinterpret_cast<int32_t*>(p);
    p += al((kMaxSup + 1) * sizeof(int32_t));
    int32_t* supcur = reinterpret_cast<int32_t*>(p);
    p += al((kMaxSup + 1) * sizeof(int32_t));
    int32_t* pstart2 = reinterpret_cast<int32_t*>(p);
    p += al((kMaxSup + 1) * sizeof(int32_t));
    void* gws = p;   // grouping of the queries by direction (group.hip)

    const uint16_t* q = reinterpret_cast<const uint16_t*>(Q);
    const uint16_t* kk = reinterpret_cast<const uint16_t*>(K);
    const uint16_t* v = reinterpret_cast<const uint16_t*>(V);
    const uint16_t* g = reinterpret_cast<const uint16_t*>(dO);
    hipError_t e;
    // The coefficient pass takes the query-heads grouped by direction once
    // there are enough pairs for the shared rows to pay for the grouping
    // (measured: 2^24 pairs and more; below, the plain order is as fast or
    // faster, 14% at 1.7M pairs in a batch of small graphs).
    QueryGroups groups{};
    if ((int64_t)pairs >= (int64_t(1) << 24)) {
        if ((e = launch_group_queries(Q, N, H, d, gws, &groups, stream)) != hipSuccess) return e;
    } else {
        int32_t* order = reinterpret_cast<int32_t*>(gws);
        groups.perm = order;
        hipLaunchKernelGGL(identity_order_kernel, dim3((unsigned)((nh + 255) / 256)), dim3(256), 0, stream, N, H,
                           order);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if ((e = launch_fill_zero(reinterpret_cast<float*>(gcnt), ((size_t)nbk + 1 + 3) / 4 * 4, stream)) != hipSuccess)
        return e;
    if ((e = launch_fill_zero(dK, (size_t)nh * d, stream)) != hipSuccess) return e;
    if ((e = launch_fill_zero(dV, (size_t)nh * d, stream)) != hipSuccess) return e;
    // pairs per counting workgroup: about 1024 workgroups, 8192 .. 65536 pairs each
    const uint32_t per = (uint32_t)std::min<size_t>(65536, std::max<size_t>(8192, (pairs / 1024 + 255) / 256 * 256));
    const unsigned cblocks = (unsigned)((pairs + per - 1) / per);
    const FastDiv divk = make_fastdiv((uint32_t)k), divh = make_fastdiv((uint32_t)H);
    hipLaunchKernelGGL(bkt_count_kernel, dim3(cblocks), dim3(256), 0, stream, idx, N, H, k, divk, divh, shift,
                       nbk, per, gcnt);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    // exclusive scan of the nbk counts; gcnt[nbk] (zero) becomes the total
    hipLaunchKernelGGL(scan_blocks_kernel, dim3((unsigned)nb), dim3(kScanBlock), 0, stream, gcnt,
                       (int64_t)nbk + 1, sums);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(scan_sums_kernel, dim3(1), dim3(kScanBlock), 0, stream, sums, nb);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(scan_apply_kernel, dim3((unsigned)nb), dim3(kScanBlock), 0, stream, gcnt,
                       (int64_t)nbk + 1, sums);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    // keep the starts, count the pieces and scan them
    hipLaunchKernelGGL(bkt_pieces_kernel, dim3((unsigned)((nbk + 1 + 255) / 256)), dim3(256), 0, stream, gcnt,
                       nbk, sstart, pstart);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(scan_blocks_kernel, dim3((unsigned)nb), dim3(kScanBlock), 0, stream, pstart,
                       (int64_t)nbk + 1, sums);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(scan_sums_kernel, dim3(1), dim3(kScanBlock), 0, stream, sums, nb);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(scan_apply_kernel, dim3((unsigned)nb), dim3(kScanBlock), 0, stream, pstart,
                       (int64_t)nbk + 1, sums);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    // the two split passes; pass 2 advances each bucket's start to its end
    const int32_t nsup = (nbk + kSupBuckets - 1) / kSupBuckets;
    hipLaunchKernelGGL(bkt_split_setup_kernel, dim3(1), dim3(64), 0, stream, sstart, nbk, nsup, supst, supcur,
                       pstart2);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    // coefficients, dQ and the interleaved copy, fused with placement pass 1
    if (d == 16)
        e = launch_coef_split<16>((int32_t)nh, stream, q, kk, v, g, idx, lse, groups.perm, N, H, k, scale, dQ, qg, shift, supcur,
                                  mid, keep, keep_scale);
    else if (d == 32)
        e = launch_coef_split<32>((int32_t)nh, stream, q, kk, v, g, idx, lse, groups.perm, N, H, k, scale, dQ, qg, shift, supcur,
                                  mid, keep, keep_scale);
    else
        e = launch_coef_split<64>((int32_t)nh, stream, q, kk, v, g, idx, lse, groups.perm, N, H, k, scale, dQ, qg, shift, supcur,
                                  mid, keep, keep_scale);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(bkt_split2_kernel, dim3((unsigned)(nsup + (pairs + kSplitChunk - 1) / kSplitChunk)), dim3(256),
                       0, stream, mid, supst, pstart2, nsup, shift, gcnt, rec);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    // at most one piece per bucket plus one per kPiece pairs; the rest exit
    const unsigned rblocks = (unsigned)(nbk + (pairs + kPiece - 1) / kPiece);
#define KMIP_BKT_REDUCE(DD, RBV)                                                                       \
    if (d == DD && rb == RBV)                                                                          \
        hipLaunchKernelGGL((bkt_reduce_kernel<DD, RBV>), dim3(rblocks), dim3(256), 0, stream, qg, rec, sstart, \
                           pstart, nbk, dK, dV);
    KMIP_BKT_REDUCE(16, 256)
    KMIP_BKT_REDUCE(16, 512)
    KMIP_BKT_REDUCE(32, 128)
    KMIP_BKT_REDUCE(32, 256)
    KMIP_BKT_REDUCE(32, 512)
    KMIP_BKT_REDUCE(64, 64)
    KMIP_BKT_REDUCE(64, 128)
    KMIP_BKT_REDUCE(64, 256)
    KMIP_BKT_REDUCE(64, 512)
#undef KMIP_BKT_REDUCE
    return hipGetLastError();
}

size_t bwd_csr_workspace_bytes(int32_t N, int32_t H, int32_t k) {
    auto al = [](size_t x) { return (x + 255) / 256 * 256; };
    const size_t nh = (size_t)N * H, pairs = nh * k;
    const size_t nb = (nh + kScanBlock - 1) / kScanBlock;
    return al(pairs * sizeof(float2)) + al(pairs * sizeof(PairRecord)) + al(nh * sizeof(int32_t)) +
           al((nb + 1) * sizeof(int32_t));
}

hipError_t launch_bwd_csr(const void* Q, const void* K, const void* V, const void* dO,
                          const int32_t* idx, const float* lse, const uint8_t* keep, float keep_scale,
                          int32_t N, int32_t H, int32_t d, int32_t dv, int32_t k, float scale, float* dQ,
                          float* dK, float* dV, void* ws, hipStream_t stream) {
    auto al = [](size_t x) { return (x + 255) / 256 * 256; };
    const int64_t nh = (int64_t)N * H;
    if (nh == 0) return hipSuccess;
    const size_t pairs = (size_t)nh * k;
    const int32_t nb = (int32_t)((nh + kScanBlock - 1) / kScanBlock);
    char* p = reinterpret_cast<char*>(ws);
    float2* coef = reinterpret_cast<float2*>(p);
    p += al(pairs * sizeof(float2));
    PairRecord* rec = reinterpret_cast<PairRecord*>(p);
    p += al(pairs * sizeof(PairRecord));
    int32_t* cnt = reinterpret_cast<int32_t*>(p);
    p += al((size_t)nh * sizeof(int32_t));
    int32_t* sums = reinterpret_cast<int32_t*>(p);

    const uint16_t* q = reinterpret_cast<const uint16_t*>(Q);
    const uint16_t* kk = reinterpret_cast<const uint16_t*>(K);
    const uint16_t* v = reinterpret_cast<const uint16_t*>(V);
    const uint16_t* g = reinterpret_cast<const uint16_t*>(dO);
    hipError_t e;
    // counts are zeroed with the float fill (same bits); n padded to 4
    if ((e = launch_fill_zero(reinterpret_cast<float*>(cnt), ((size_t)nh + 3) / 4 * 4, stream)) != hipSuccess) return e;
    if ((e = launch_fill_zero(dK, (size_t)nh * d, stream)) != hipSuccess) return e;
    if ((e = launch_fill_zero(dV, (size_t)nh * dv, stream)) != hipSuccess) return e;
    const unsigned team_blocks = (unsigned)((nh + 15) / 16);
    bool launched = false;
#define KMIP_CSR_COEF(DD, DVV)                                                                          \
    if (d == DD && dv == DVV) {                                                                         \
        launch_coef<DD, DVV>(team_blocks, stream, q, kk, v, g, idx, lse, N, H, k, scale, dQ, coef, nullptr, \
                             keep, keep_scale);                                                          \
        launched = true;                                                                                \
    }
#define KMIP_CSR_COEF_D(DD) KMIP_CSR_COEF(DD, 16) KMIP_CSR_COEF(DD, 32) KMIP_CSR_COEF(DD, 64) KMIP_CSR_COEF(DD, 128)
    KMIP_CSR_COEF_D(16)
    KMIP_CSR_COEF_D(32)
    KMIP_CSR_COEF_D(64)
    KMIP_CSR_COEF_D(128)
#undef KMIP_CSR_COEF_D
#undef KMIP_CSR_COEF
    if (!launched) return hipErrorInvalidValue;
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const unsigned qh_blocks = (unsigned)((nh + 255) / 256);
    hipLaunchKernelGGL(csr_count_kernel<false>, dim3(qh_blocks), dim3(256), 0, stream, idx, coef, N, H,
                       k, cnt, rec);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(scan_blocks_kernel, dim3((unsigned)nb), dim3(kScanBlock), 0, stream, cnt,
                       (int64_t)nh, sums);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(scan_sums_kernel, dim3(1), dim3(kScanBlock), 0, stream, sums, nb);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(scan_apply_kernel, dim3((unsigned)nb), dim3(kScanBlock), 0, stream, cnt,
                       (int64_t)nh, sums);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(csr_count_kernel<true>, dim3(qh_blocks), dim3(256), 0, stream, idx, coef, N, H,
                       k, cnt, rec);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    // one team per kChunk/4 sorted pairs, 16 teams per block; the grid covers
    // every pair slot, teams past the total exit at once
    const unsigned red_blocks = (unsigned)((pairs + kChunk * 4 - 1) / (kChunk * 4));
    const int32_t* total = sums + nb;
#define KMIP_CSR_REDUCE(DD, DVV)                                                                        \
    if (d == DD && dv == DVV)                                                                           \
        hipLaunchKernelGGL((csr_reduce_kernel<DD, DVV>), dim3(red_blocks), dim3(256), 0, stream, q, g, rec, \
                           total, dK, dV);
#define KMIP_CSR_REDUCE_D(DD) \
    KMIP_CSR_REDUCE(DD, 16) KMIP_CSR_REDUCE(DD, 32) KMIP_CSR_REDUCE(DD, 64) KMIP_CSR_REDUCE(DD, 128)
    KMIP_CSR_REDUCE_D(16)
    KMIP_CSR_REDUCE_D(32)
    KMIP_CSR_REDUCE_D(64)
    KMIP_CSR_REDUCE_D(128)
#undef KMIP_CSR_REDUCE_D
#undef KMIP_CSR_REDUCE
    return hipGetLastError();
}

}  // namespace kmip
