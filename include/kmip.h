/*
 * kmip.h -- C ABI of the MI355X (gfx950) k-MIP self-attention library.
 *
 * k-Maximum Inner Product attention (arXiv 2604.03815, Section 3.1, Eq. 1;
 * Algorithm 1 in Appendix E): for every query node i and head h, score i
 * against every key node j of the query's own graph (s_ij = q_i . k_j),
 * keep the k largest scores, take a softmax over the k kept scores times
 * `scale`, and sum the matching value rows.  The N x N score matrix is never
 * stored (the symbolic-matrix idea of Appendix F): memory is linear in N.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Q, K, V, dOut: bfloat16, device memory, layout [N, H, d] row-major
 *    (node-major: element (i, h, t) at ((i * H) + h) * d + t).
 *  - out, dQ, dK, dV: float32, device memory, layout [N, H, d].
 *  - topk_idx: int32, device memory, [N, H, k].  Global 0-based node ids,
 *    ordered by (score descending, node id ascending).  When the query's
 *    graph has n < k nodes, slots n..k-1 hold -1.
 *  - lse: float32, device memory, [N, H]: natural log of
 *    sum_{j kept} exp(scale * s_ij).
 *  - graph_offsets: HOST memory, int32 [num_graphs + 1], o_0 = 0,
 *    non-decreasing, o_G = N.  Query i of graph g attends only to keys in
 *    [o_g, o_{g+1}) (block-diagonal batching of many graphs).  NULL means a
 *    single graph of N nodes (num_graphs is then ignored).  Empty graphs are
 *    allowed.  With several graphs the library builds a work list on the
 *    host and uploads it on the caller's stream through pinned host memory
 *    that it keeps (two buffers per device, grown on demand, until the
 *    process ends), so that the call does not wait for the stream; the
 *    offsets array may be reused as soon as the call returns.
 *  - Ties between equal scores go to the lower node id.  The query's own
 *    key is a candidate.  `scale` must be finite and > 0; selection uses the
 *    raw scores, which for scale > 0 is the same as the scaled scores.
 *  - Supported sizes: d in {16, 32, 64, 128}; 1 <= k <= KMIP_MAX_K (512)
 *    for d <= 64 and 1 <= k <= KMIP_MAX_K_WIDE (128) for d = 128; H >= 1;
 *    0 <= N < 2^31 and N * H * max(d, k) < 2^31.  (The bound on N * H * k
 *    is also what keeps node ids below 2^(32 - ceil(log2 k)), the room the
 *    select kernel's on-chip trees leave for an index.)  The fastest paths
 *    are those of d <= 64 and k <= 128: the direction grouping and the key
 *    order with bounds that let the select kernel skip key blocks are built
 *    for d <= 64 only, and a larger k gives the kernel larger trees in LDS
 *    (fewer resident waves).
 *  - stream: a hipStream_t (NULL = the default stream).  Every call is
 *    asynchronous on `stream`; the caller synchronises.
 *  - Ownership: the caller allocates every buffer (inputs, outputs and the
 *    workspace); the library allocates no device memory and keeps no state
 *    between calls (apart from kmip_fwd_noalloc's fixed per-device array,
 *    which holds no state from one call to the next).  Outputs are
 *    overwritten, never accumulated.
 *  - Errors: arguments are validated on the host before any launch; on
 *    error nothing is launched and outputs are untouched.  Index entries
 *    read by kmip_attend / kmip_bwd that fall outside [0, N) are treated as
 *    empty slots, never dereferenced.  NaN or Inf in the inputs, or scores
 *    that overflow float32, give undefined (but memory-safe) results.
 *    No exception crosses the ABI.
 */
#ifndef KMIP_H_
#define KMIP_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    KMIP_OK = 0,
    KMIP_ERR_INVALID_ARG = 1, /* null buffer, bad size, bad offsets, bad scale */
    KMIP_ERR_UNSUPPORTED = 2, /* d, d_V, k or variant outside the compiled set */
    KMIP_ERR_WORKSPACE = 3,   /* workspace missing or smaller than required */
    KMIP_ERR_HIP = 4          /* a HIP launch or copy failed; see kmip_last_error() */
} kmip_status_t;

#define KMIP_MAX_K 512      /* largest k for d <= 64 */
#define KMIP_MAX_K_WIDE 128 /* largest k for d = 128 */

/*
 * Bytes of device workspace kmip_topk / kmip_fwd need for these sizes
 * (0 if the sizes are invalid).  Holds a tiled copy of K and, for more than
 * one graph, the work list; for a single graph of at least 8192 nodes, the
 * grouping of the queries by direction and the stored order of the keys
 * with the bounds the kernel uses to skip key blocks (linear in N).
 */
size_t kmip_topk_workspace_size(int64_t N, int32_t H, int32_t d, int32_t k, int32_t num_graphs);

/*
 * Score + select (Algorithm 1: SymbolicMultiply followed by RowwiseTopK;
 * Appendix F).  For every query and head, streams the keys of the query's
 * graph, forms bf16 score tiles on the matrix cores with fp32 accumulation,
 * and keeps the k best (score, index) pairs on chip.
 *   out: topk_idx [N, H, k].
 *   workspace: device memory of at least kmip_topk_workspace_size() bytes,
 *   256-byte aligned; its contents on entry do not matter.
 */
kmip_status_t kmip_topk(const void* Q, const void* K, const int32_t* graph_offsets,
                        int32_t num_graphs, int64_t N, int32_t H, int32_t d, int32_t k,
                        int32_t* topk_idx, void* workspace, size_t workspace_bytes,
                        void* stream);

/*
 * kmip_topk, recording two events around the score+select kernel alone (not
 * the pre-passes that group the queries and order the keys), for callers
 * that time that kernel.
 *   select_start, select_stop: hipEvent_t handles created by the caller, or
 *   NULL to record nothing; recorded on `stream` right before and right after
 *   the kernel's launch.  On an error return neither is recorded.
 */
kmip_status_t kmip_topk_with_events(const void* Q, const void* K, const int32_t* graph_offsets,
                                    int32_t num_graphs, int64_t N, int32_t H, int32_t d, int32_t k,
                                    int32_t* topk_idx, void* workspace, size_t workspace_bytes,
                                    void* stream, void* select_start, void* select_stop);

/*
 * Score + select with low-precision candidate scoring (the paper names
 * FP16/INT8 scoring on matrix cores as its next step: Appendix, comparison
 * with FlashAttention, closing paragraph), for one graph (no
 * graph_offsets) and k <= 32.  Same result as kmip_topk, order included:
 *   1. Q and K are quantised to int8 with power-of-two scales (one per head
 *      for K, one per query), and every key is scored exactly in int32 on
 *      the matrix cores (v_mfma_i32_32x32x32_i8);
 *   2. from the quantisation errors, a bound E + delta on the gap between
 *      those scores and kmip_topk's fp32 scores gives each query an integer
 *      threshold that every key of its exact top-k clears (ties included),
 *      and a second int8 pass lists the keys that clear it (at most 1024 a
 *      query);
 *   3. the listed keys are scored again with kmip_topk's bf16 MFMA and the
 *      k best taken by (score descending, node id ascending).
 *   Queries whose list would overflow (data whose top-k scores lie closer
 *   together than the int8 error) have their blocks of 32 queries redone by
 *   kmip_topk's select kernel on the device, so the result never depends on
 *   the data.  k > 32 returns KMIP_ERR_UNSUPPORTED.
 *   redone: device int32, or NULL: receives (on the stream) the number of
 *   query blocks of 32 that the select kernel redid.
 *   workspace: kmip_topk_prefilter_workspace_size() bytes (0 if the sizes
 *   are not taken), 256-byte aligned; about 4 KB per query-head.
 */
size_t kmip_topk_prefilter_workspace_size(int64_t N, int32_t H, int32_t d, int32_t k);
kmip_status_t kmip_topk_prefilter(const void* Q, const void* K, int64_t N, int32_t H, int32_t d, int32_t k,
                                  int32_t* topk_idx, int32_t* redone, void* workspace, size_t workspace_bytes,
                                  void* stream);

/*
 * Gather-softmax-aggregate (Algorithm 1: GatherRows, softmax over the k kept
 * scores divided by sqrt(d_K) -- here times `scale` -- and the einsum
 * nk,nkv->nv).  Recomputes the k kept scores in fp32 from Q and the gathered
 * K rows, then sums the gathered V rows.  Needs no workspace.
 *   in:  topk_idx [N, H, k] (e.g. from kmip_topk; -1 marks an empty slot).
 *   out: out [N, H, d], lse [N, H].  A query with no valid slot gets
 *        out = 0 and lse = -inf.
 */
kmip_status_t kmip_attend(const void* Q, const void* K, const void* V, int64_t N, int32_t H,
                          int32_t d, int32_t k, float scale, const int32_t* topk_idx,
                          float* out, float* lse, void* stream);

/* kmip_topk followed by kmip_attend on the same stream; same workspace as kmip_topk. */
size_t kmip_fwd_workspace_size(int64_t N, int32_t H, int32_t d, int32_t k, int32_t num_graphs);
kmip_status_t kmip_fwd(const void* Q, const void* K, const void* V, const int32_t* graph_offsets,
                       int32_t num_graphs, int64_t N, int32_t H, int32_t d, int32_t k,
                       float scale, float* out, int32_t* topk_idx, float* lse,
                       void* workspace, size_t workspace_bytes, void* stream);

/*
 * Extended forward entry points for training use:
 *  - value rows of their own width (Section 3.1: W_Q and W_K project to
 *    d_K dimensions, W_V to d_V): Q and K are [N, H, d] with d = d_K, which
 *    alone decides the selection; V and out are [N, H, dv] with
 *    dv = d_V in {16, 32, 64, 128};
 *  - attention dropout (the experimental details list an attention-dropout
 *    rate): keep is uint8 [N, H, k] device memory aligned with the topk_idx
 *    slots, drawn by the caller (nonzero keeps the slot); the kept weights
 *    are multiplied by 1 / (1 - drop_rate), the dropped ones by 0 (inverted
 *    dropout).  lse stays that of the softmax before dropout.  keep = NULL
 *    with drop_rate = 0 is no dropout; a drop_rate outside [0, 1), or > 0
 *    without keep, is KMIP_ERR_INVALID_ARG.
 * kmip_attend / kmip_fwd are the case dv = d, keep = NULL.  Same workspace
 * as kmip_topk; N * H * dv < 2^31.
 */
kmip_status_t kmip_attend_ex(const void* Q, const void* K, const void* V, int64_t N, int32_t H,
                             int32_t d, int32_t dv, int32_t k, float scale, const int32_t* topk_idx,
                             const uint8_t* keep, float drop_rate, float* out, float* lse, void* stream);
kmip_status_t kmip_fwd_ex(const void* Q, const void* K, const void* V, const int32_t* graph_offsets,
                          int32_t num_graphs, int64_t N, int32_t H, int32_t d, int32_t dv, int32_t k,
                          float scale, const uint8_t* keep, float drop_rate, float* out, int32_t* topk_idx,
                          float* lse, void* workspace, size_t workspace_bytes, void* stream);

/*
 * kmip_fwd_ex, recording caller events for timing: select_start and
 * select_stop as kmip_topk_with_events does (around the score+select
 * kernel alone), attend_start right before the aggregate.  Each may be NULL
 * to record nothing.  In every kmip_fwd* call on one graph that the library
 * groups by direction (at least 8192 nodes, d <= 64) the aggregate takes
 * the query-heads in that grouped order, so that the queries of a
 * workgroup share their keys' rows; results do not depend on the order.
 */
kmip_status_t kmip_fwd_ex_with_events(const void* Q, const void* K, const void* V, const int32_t* graph_offsets,
                                      int32_t num_graphs, int64_t N, int32_t H, int32_t d, int32_t dv, int32_t k,
                                      float scale, const uint8_t* keep, float drop_rate, float* out,
                                      int32_t* topk_idx, float* lse, void* workspace, size_t workspace_bytes,
                                      void* stream, void* select_start, void* select_stop, void* attend_start);

/*
 * Backward with the forward's index set held fixed (Section 3.1, last
 * paragraph, and Appendix E, last paragraph: the top-k indices are reused,
 * so only the k selected pairs of each query carry gradient).  With p_j the
 * softmax weights of query i (recomputed from Q, K, topk_idx and lse):
 *   dp_j = dOut_i . v_j,  D_i = sum_j p_j dp_j,  g_j = p_j (dp_j - D_i),
 *   dQ_i = scale sum_j g_j k_j,  dK_j += scale g_j q_i,  dV_j += p_j dOut_i.
 *   in:  dOut bf16 [N, H, d]; topk_idx [N, H, k] and lse [N, H] as written
 *        by the forward.
 *   out: dQ, dK, dV float32 [N, H, d], overwritten.
 *
 * Parameters compared with the forward's: there is no graph_offsets,
 * num_graphs or out.  The saved indices are global node ids that already
 * lie in their query's graph, so the batch structure is not needed again;
 * and D_i = sum_j p_j dp_j comes from the dp_j that g_j needs anyway, so
 * the forward's out (whose dot product with dOut_i is the same D_i) is not
 * read.  The order is (inputs, saved tensors, sizes, scale, outputs,
 * variant, workspace, stream).
 *
 *   variant (kmip_bwd_variant_t): how dK and dV are summed over the queries
 *            that selected a key.  All use fp32 atomics somewhere, so the
 *            summation order is not fixed and results may differ in the
 *            last bits from call to call.
 *            KMIP_BWD_ATOMIC: every selected pair adds its rows with
 *                atomics;
 *            KMIP_BWD_SEGMENTED: the pairs are counting-sorted by key row
 *                and each key's run is summed in registers, one atomic per
 *                run piece of 256 pairs;
 *            KMIP_BWD_BUCKETED: the pairs are counting-sorted by buckets of
 *                consecutive key rows (j*H + h), 4096/d of them, doubled up
 *                to 512 while N*H would need more than 8192 buckets; each
 *                bucket's records are sorted by key row in LDS, at most 8192
 *                at a time, and reduced as in SEGMENTED; needs
 *                N*H <= 8192*512, d <= 64 and k <= 128 (else
 *                KMIP_ERR_UNSUPPORTED and workspace size 0);
 *            KMIP_BWD_KEY_AGGREGATED: queries are grouped by direction, each
 *                workgroup of 256 queries sums its pairs per key in LDS and
 *                adds each key's sums once;
 *            KMIP_BWD_AUTO: BUCKETED where it is supported, else SEGMENTED;
 *            any other value: KMIP_ERR_UNSUPPORTED.
 *   workspace: kmip_bwd_workspace_size(variant) bytes, 256-byte aligned
 *              (0 for KMIP_BWD_ATOMIC, which accepts NULL); too small or
 *              misaligned -> KMIP_ERR_WORKSPACE.
 */
typedef enum {
    KMIP_BWD_AUTO = 0,
    KMIP_BWD_ATOMIC = 1,
    KMIP_BWD_SEGMENTED = 2,
    KMIP_BWD_BUCKETED = 3,
    KMIP_BWD_KEY_AGGREGATED = 4
} kmip_bwd_variant_t;

size_t kmip_bwd_workspace_size(int64_t N, int32_t H, int32_t d, int32_t k, int32_t variant);
kmip_status_t kmip_bwd(const void* Q, const void* K, const void* V, const void* dOut,
                       const int32_t* topk_idx, const float* lse, int64_t N, int32_t H,
                       int32_t d, int32_t k, float scale, float* dQ, float* dK, float* dV,
                       int32_t variant, void* workspace, size_t workspace_bytes, void* stream);

/*
 * kmip_bwd for the extended forward: value rows of width dv = d_V in
 * {16, 32, 64, 128} (V, dOut bf16 [N, H, dv] and dV float32 [N, H, dv]; Q, K,
 * dQ, dK stay [N, H, d]; dp_j = dOut_i . v_j runs over the dv value
 * dimensions) and the forward's dropout draws keep / drop_rate (with
 * f_j = 1/(1 - drop_rate) for a kept slot and 0 for a dropped one, dV_j gets
 * p_j f_j dOut_i and f_j dp_j replaces dp_j in D_i and g_j).
 * KMIP_BWD_BUCKETED needs dv == d (else KMIP_ERR_UNSUPPORTED and workspace
 * size 0): its interleaved copy of q_i and dOut_i assumes equal widths;
 * KMIP_BWD_AUTO then picks KMIP_BWD_SEGMENTED.  kmip_bwd and
 * kmip_bwd_workspace_size are the case dv = d, keep = NULL.
 */
size_t kmip_bwd_ex_workspace_size(int64_t N, int32_t H, int32_t d, int32_t dv, int32_t k, int32_t variant);
kmip_status_t kmip_bwd_ex(const void* Q, const void* K, const void* V, const void* dOut,
                          const int32_t* topk_idx, const float* lse, const uint8_t* keep, float drop_rate,
                          int64_t N, int32_t H, int32_t d, int32_t dv, int32_t k, float scale, float* dQ,
                          float* dK, float* dV, int32_t variant, void* workspace, size_t workspace_bytes,
                          void* stream);

/*
 * Forward (kmip_fwd) of one graph without a caller workspace and without
 * allocating anything, for callers that cannot allocate device or pinned
 * memory during the call: code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation.
 *   The score + select pass keeps its working data (tiled keys, query
 *   grouping, key order, work counters) in a fixed device array of
 *   KMIP_NOALLOC_SCRATCH_BYTES bytes inside this library, one per GPU the
 *   library runs on, held until the process ends.  Its device address is
 *   looked up on the first call on each device.
 *   Arguments, layouts and results are kmip_fwd's for graph_offsets = NULL:
 *   Q, K, V bf16 [N, H, d]; out float32 [N, H, d], topk_idx int32 [N, H, k],
 *   lse float32 [N, H], all caller-owned device memory.  Block-diagonal
 *   batches are not taken (their work list is uploaded through pinned host
 *   memory that kmip_fwd allocates): use kmip_fwd for them.
 *   Sizes whose kmip_fwd_workspace_size(N, H, d, k, 1) exceeds
 *   KMIP_NOALLOC_SCRATCH_BYTES return KMIP_ERR_UNSUPPORTED (N = 500,000,
 *   H = 4, d = 16, k = 32 needs 223 MiB) before anything is launched.
 *   Every call on one GPU shares that GPU's array: calls that overlap on
 *   one GPU (on different streams, or from different host threads without
 *   ordering) race and give undefined results.  Calls ordered on one
 *   stream are safe; each call clears the counters it reads.
 */
#define KMIP_NOALLOC_SCRATCH_BYTES (256u * 1024u * 1024u)
kmip_status_t kmip_fwd_noalloc(const void* Q, const void* K, const void* V, int64_t N, int32_t H,
                               int32_t d, int32_t k, float scale, float* out, int32_t* topk_idx,
                               float* lse, void* stream);

/* Static description of a status code. */
const char* kmip_status_string(kmip_status_t status);

/* Detail of the last error on the calling host thread ("" if none). */
const char* kmip_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* KMIP_H_ */
