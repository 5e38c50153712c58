// Internal declarations shared by the kmip HIP sources (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kmip.h"

namespace kmip {

// Zero tiles appended to each head of the tiled key buffer, so that key
// prefetches running past a head's last tile stay in bounds (at least the
// prefetch depth plus one).
constexpr int kPadTiles = 16;

// Number of XCDs of MI355X; workgroups are dispatched to them round-robin.
constexpr int kNumXcd = 8;

// Device scratch the select kernel needs for its work counters and pacers.
constexpr size_t kSelectCounterBytes = 512;

// One unit of score+select work: a run of up to 32*QB queries of one graph
// and the key range of that graph.
struct Task {
    int32_t q_begin;
    int32_t q_count;
    int32_t key_lo;
    int32_t key_hi;
};

// ---- launchers (host side); each returns hipSuccess or the launch error ----

// Tiles K [N,H,d] bf16 into the matrix-core operand order: for head h and key
// tile t (32 positions), chunk c of 16 dims, lane l holds 8 bf16 of the key at
// position p = 32t + l%32, dims 16c + 8(l/32) .. +8.  Position p holds key
// perm[h][p] (key p when perm is NULL); positions >= N are zero; each head has
// ntiles + kPadTiles tiles.  rows, when not NULL, holds those keys' rows
// already in position order, head-major [H][N][d], and is read instead.
hipError_t launch_pack_k(const void* K, const int32_t* perm, const uint16_t* rows, void* kp, int32_t N,
                         int32_t H, int32_t d, int32_t ntiles, hipStream_t stream);

// Stored key order with superblock bounds (keyorder.hip): the leaf order of
// a balanced space-partitioning tree whose leaves are superblocks of
// kSuperTiles tiles, each with a ball bound.
constexpr int kSuperTiles = 8;
// Net votes (items finding most superblocks needed, minus the others) at
// which a head's select items stop forming masks and scan every superblock.
constexpr int kDenseVotes = 16;
// Net votes (seeded items whose lower-bound pass raised no threshold, minus
// the others) at which a head's seeded items skip that pass.
constexpr int kLowerVotes = 16;

// Device arrays of a key order:
//   perm   [H][N]  key stored at each position;
//   bounds [H][ctiles][d/16 + 1][64] uint4: bound tiles, superblock s in
//          tile s / 32, row s % 32, in the key-tile operand layout: chunks
//          0 .. d/16-1 the bf16 center, chunk d/16 the radius R (bf16, rounded
//          up) in dim 0;
//   votes  [2H] dense-mode votes, then lower-bound-pass votes (zero before
//          the select launch).
//   wbounds [H][wctiles][d/16 + 1][64] uint4: window tiles, the same kind of
//          ball bound for each window of 64 superblocks (window w in tile
//          w / 32, row w % 32).
struct KeyOrder {
    const int32_t* perm;
    const uint16_t* rows;   // key rows in the stored order, head-major [H][N][d]
    const uint4* bounds;
    int32_t* votes;
    int32_t ctiles;
    const uint4* wbounds;
    int32_t wctiles;
};

// Bound tiles per head for ntiles key tiles: two per 64 superblocks.
int32_t key_order_ctiles(int32_t ntiles);
// Window tiles per head for ctiles bound tiles: two per 64 windows.
int32_t key_order_wctiles(int32_t ctiles);
size_t key_order_workspace_bytes(int32_t N, int32_t H, int32_t d);
hipError_t launch_key_order(const void* K, int32_t N, int32_t H, int32_t d, int32_t ntiles, void* ws,
                            KeyOrder* out, hipStream_t stream);

// Shape of one select wave: query blocks of 32 and candidate-buffer slots
// per lane and block, {2, 4} or {1, 8}.
struct SelectShape {
    int32_t qb;
    int32_t slots;
};

// Queries grouped by direction (group.hip), all arrays in device memory:
//   perm     [H][N]  query processed at position p of head h;
//   label    [H][N]  reference direction nearest to query i of head h;
//   seed_ref [H][kGroupCenters]  0, or 1 + a query id of that label whose
//            finished top-k row other queries of the label may seed from
//            (zero before the select launch).
struct QueryGroups {
    const int32_t* perm;
    const uint16_t* label;
    int32_t* seed_ref;
};

// Score + select.  kp: the tiled keys (launch_pack_k).  groups: NULL
// (identity order, no seeding; always so for a block-diagonal batch), or the
// grouping of the queries.  keys: NULL (every tile scanned), or the stored
// key order kp was packed in, with its bounds.  K: the keys in their own
// layout (seed rows are gathered from it).  work_ctr: kSelectCounterBytes of device scratch, 8-byte aligned
// (per-XCD item counters and stream pacers, zeroed here).  ev_start /
// ev_stop: events recorded right before and after the kernel, or NULL.
hipError_t launch_select(const void* kp, const void* Q, const void* K, const Task* tasks,
                         const QueryGroups* groups, const KeyOrder* keys, int32_t ntasks, int32_t N,
                         int32_t H, int32_t d, int32_t k, int32_t ntiles, SelectShape shape,
                         int32_t* work_ctr, int32_t* topk_idx, hipStream_t stream,
                         hipEvent_t ev_start, hipEvent_t ev_stop);

// Bytes of LDS one select workgroup uses.
size_t select_lds_bytes(int32_t k, SelectShape shape);

// Graphs of a block-diagonal batch with at most this many nodes go to the
// small-graph select (small_select.hip), which keeps a whole graph's scores
// of 32 queries in LDS.
constexpr int kSmallGraph = 480;

// Score + select for tasks of at most 32 queries whose graphs hold at most
// kSmallGraph nodes (same results as launch_select).
hipError_t launch_small_select(const void* kp, const void* Q, const Task* tasks, int32_t ntasks, int32_t N,
                               int32_t H, int32_t d, int32_t k, int32_t ntiles, int32_t* topk_idx,
                               hipStream_t stream);

// Query grouping by direction (group.hip): reference directions per head.
constexpr int kGroupCenters = 256;

// Workspace bytes launch_group_queries needs.
size_t group_workspace_bytes(int32_t N, int32_t H, int32_t d);

// Groups the queries of each head by direction into ws and describes the
// result in *out.
// The query order [H][N] a grouping workspace holds after
// launch_group_queries (the same address QueryGroups::perm was given).
const int32_t* group_perm_in(const void* ws, int32_t N, int32_t H, int32_t d);
hipError_t launch_group_queries(const void* Q, int32_t N, int32_t H, int32_t d, void* ws,
                                QueryGroups* out, hipStream_t stream);

// Gather-softmax-aggregate: Q, K [N,H,d] (d = d_K), V and out [N,H,dv]
// (dv = d_V), each in {16, 32, 64}.
// keep / keep_scale: attention dropout draws uint8 [N,H,k] and 1/(1 - rate),
// or nullptr (no dropout), for this launcher and the backward ones.
hipError_t launch_attend(const void* Q, const void* K, const void* V, const int32_t* idx,
                         const uint8_t* keep, float keep_scale, int32_t N, int32_t H, int32_t d, int32_t dv,
                         int32_t k, float scale, const int32_t* perm, float* out, float* lse,
                         hipStream_t stream);

// The backward launchers take the query/key width d and the value width dv
// (each in {16, 32, 64}); the bucketed one needs dv == d.
hipError_t launch_bwd_atomic(const void* Q, const void* K, const void* V, const void* dO,
                             const int32_t* idx, const float* lse, const uint8_t* keep, float keep_scale,
                             int32_t N, int32_t H, int32_t d, int32_t dv, int32_t k, float scale, float* dQ,
                             float* dK, float* dV, hipStream_t stream);

// Backward with key-aggregated scatter; ws holds bwd_agg_workspace_bytes().
size_t bwd_agg_workspace_bytes(int32_t N, int32_t H, int32_t d);
hipError_t launch_bwd_agg(const void* Q, const void* K, const void* V, const void* dO,
                          const int32_t* idx, const float* lse, const uint8_t* keep, float keep_scale,
                          int32_t N, int32_t H, int32_t d, int32_t dv, int32_t k, float scale, float* dQ,
                          float* dK, float* dV, void* ws, hipStream_t stream);

// Backward with a key-sorted segmented reduction (backward_csr.hip); ws
// holds bwd_csr_workspace_bytes().
size_t bwd_csr_workspace_bytes(int32_t N, int32_t H, int32_t k);
hipError_t launch_bwd_csr(const void* Q, const void* K, const void* V, const void* dO,
                          const int32_t* idx, const float* lse, const uint8_t* keep, float keep_scale,
                          int32_t N, int32_t H, int32_t d, int32_t dv, int32_t k, float scale, float* dQ,
                          float* dK, float* dV, void* ws, hipStream_t stream);

// Backward with pairs bucketed by blocks of key rows and summed in LDS
// (backward_csr.hip); supported for d <= 64 and k <= 128 while
// N * H / (4096 / d) <= 8192.
bool bwd_bucket_supported(int32_t N, int32_t H, int32_t d, int32_t k);
size_t bwd_bucket_workspace_bytes(int32_t N, int32_t H, int32_t d, int32_t k);
hipError_t launch_bwd_bucket(const void* Q, const void* K, const void* V, const void* dO,
                             const int32_t* idx, const float* lse, const uint8_t* keep, float keep_scale,
                             int32_t N, int32_t H, int32_t d, int32_t k, float scale, float* dQ, float* dK,
                             float* dV, void* ws, hipStream_t stream);

hipError_t launch_fill_zero(float* p, size_t n, hipStream_t stream);

// Int8 prefilter with a provable bound and exact re-rank (prefilter.hip), for
// one graph and k <= 32.  Candidates listed per query-head (two halves).
constexpr int kPrefilterCap = 1024;
constexpr int kPrefilterMaxK = 32;
// Bytes of the int8 key tiles: H x (ceil(N/32) + kPadTiles) tiles of
// ceil(d/32) chunks of 1 KB.
size_t prefilter_tile_bytes(int32_t N, int32_t H, int32_t d);
// Writes topk_idx for every query-head whose candidate list fits; the query
// blocks of the others are listed in fb_tasks[0 .. *fb_count) (the rest of
// fb_tasks, ceil(N/32) entries, holds zero-query tasks) for the select
// kernel to redo.  hstat: 4 H words; cand: N H kPrefilterCap ints; ccount:
// 2 N H ints; flags: H ceil(N/32) ints.
hipError_t launch_prefilter(const void* K, const void* Q, int32_t N, int32_t H, int32_t d, int32_t k,
                            uint32_t* hstat, uint4* kp8, int32_t* cand, int32_t* ccount, int32_t* flags,
                            int32_t* fb_count, Task* fb_tasks, int32_t* topk_idx, hipStream_t stream);

// Sets the calling thread's kmip_last_error() text (printf-style) and
// returns s.
kmip_status_t record_error(kmip_status_t s, const char* fmt, ...);

}  // namespace kmip
