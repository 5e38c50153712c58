// Host side of the kmip C ABI (declared in include/kmip.h): argument
// validation, workspace layout, the block-diagonal work list and launches.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "kmip.h"
#include "kmip_internal.h"

namespace {
thread_local std::string g_last_error;
}  // namespace

namespace kmip {

kmip_status_t record_error(kmip_status_t s, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return s;
}

}  // namespace kmip

namespace {

using kmip::record_error;

kmip_status_t ok() {
    g_last_error.clear();
    return KMIP_OK;
}

kmip_status_t hip_fail(hipError_t e, const char* what) {
    return record_error(KMIP_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

constexpr size_t kAlign = 256;

// Pinned host staging for the block-diagonal work list, so that its upload
// is an asynchronous copy (a copy from pageable memory blocks the caller
// until the stream reaches it).  Two buffers per device, used in turn; a
// buffer is refilled only after the copy that last read it has completed
// (an event recorded behind that copy).  Kept until the process ends.
struct Staging {
    void* buf[2] = {nullptr, nullptr};
    size_t cap[2] = {0, 0};
    hipEvent_t ev[2] = {nullptr, nullptr};
    int next = 0;
};
constexpr int kMaxDevices = 64;
std::mutex g_stage_mu;
Staging g_stage[kMaxDevices];

// Copies `bytes` from host `src` to device `dst` on `stream` through the
// calling device's staging buffers.
hipError_t upload_async(void* dst, const void* src, size_t bytes, hipStream_t stream) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipMemcpyAsync(dst, src, bytes, hipMemcpyHostToDevice, stream);
    std::lock_guard<std::mutex> lock(g_stage_mu);
    Staging& st = g_stage[dev];
    const int i = st.next;
    st.next ^= 1;
    if (st.ev[i] == nullptr) {
        if ((e = hipEventCreateWithFlags(&st.ev[i], hipEventDisableTiming)) != hipSuccess) return e;
    } else if ((e = hipEventSynchronize(st.ev[i])) != hipSuccess) {
        return e;
    }
    if (st.cap[i] < bytes) {
        if (st.buf[i] != nullptr && (e = hipHostFree(st.buf[i])) != hipSuccess) return e;
        st.buf[i] = nullptr;
        st.cap[i] = 0;
        const size_t cap = std::max<size_t>(bytes, 64 * 1024);
        if ((e = hipHostMalloc(&st.buf[i], cap, hipHostMallocDefault)) != hipSuccess) return e;
        st.cap[i] = cap;
    }
    std::memcpy(st.buf[i], src, bytes);
    if ((e = hipMemcpyAsync(dst, st.buf[i], bytes, hipMemcpyHostToDevice, stream)) != hipSuccess) return e;
    return hipEventRecord(st.ev[i], stream);
}

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Sizes shared by all entry points.
kmip_status_t check_sizes(int64_t N, int32_t H, int32_t d, int32_t k) {
    if (N < 0 || N >= (int64_t(1) << 31)) return record_error(KMIP_ERR_INVALID_ARG, "N=%lld out of range", (long long)N);
    if (H < 1) return record_error(KMIP_ERR_INVALID_ARG, "H=%d must be >= 1", H);
    if (k < 1) return record_error(KMIP_ERR_INVALID_ARG, "k=%d must be >= 1", k);
    if (d != 16 && d != 32 && d != 64 && d != 128)
        return record_error(KMIP_ERR_UNSUPPORTED, "d=%d not in {16, 32, 64, 128}", d);
    const int32_t kmax = d == 128 ? KMIP_MAX_K_WIDE : KMIP_MAX_K;
    if (k > kmax) return record_error(KMIP_ERR_UNSUPPORTED, "k=%d exceeds %d for d=%d", k, kmax, d);
    const int64_t wide = N * (int64_t)H * std::max<int64_t>(d, k);
    if (wide >= (int64_t(1) << 31)) return record_error(KMIP_ERR_INVALID_ARG, "N*H*max(d,k) >= 2^31");
    return KMIP_OK;
}

// The value width, besides the sizes check_sizes covers.
kmip_status_t check_value_width(int64_t N, int32_t H, int32_t dv) {
    if (dv != 16 && dv != 32 && dv != 64 && dv != 128)
        return record_error(KMIP_ERR_UNSUPPORTED, "d_V=%d not in {16, 32, 64, 128}", dv);
    if (N * (int64_t)H * dv >= (int64_t(1) << 31)) return record_error(KMIP_ERR_INVALID_ARG, "N*H*d_V >= 2^31");
    return KMIP_OK;
}

// Finite test on the bits: the sources are built with -fno-honor-nans (for
// the kernels' max3 chains), under which std::isfinite may assume no NaN.
bool finite_bits(float x) {
    uint32_t b;
    std::memcpy(&b, &x, sizeof(b));
    return (b & 0x7F800000u) != 0x7F800000u;
}

// Attention dropout: a rate in [0, 1); keep draws are needed for a rate > 0.
kmip_status_t check_dropout(const uint8_t* keep, float rate) {
    if (!finite_bits(rate) || rate < 0.0f || rate >= 1.0f)
        return record_error(KMIP_ERR_INVALID_ARG, "drop_rate must lie in [0, 1)");
    if (keep == nullptr && rate != 0.0f) return record_error(KMIP_ERR_INVALID_ARG, "drop_rate > 0 needs keep draws");
    return KMIP_OK;
}

kmip_status_t check_scale(float scale) {
    if (!finite_bits(scale) || !(scale > 0.0f)) return record_error(KMIP_ERR_INVALID_ARG, "scale must be finite and > 0");
    return KMIP_OK;
}

kmip_status_t check_offsets(const int32_t* off, int32_t G, int64_t N) {
    if (off == nullptr) return KMIP_OK;
    if (G < 1) return record_error(KMIP_ERR_INVALID_ARG, "num_graphs=%d must be >= 1 with offsets", G);
    if (off[0] != 0) return record_error(KMIP_ERR_INVALID_ARG, "graph_offsets[0]=%d must be 0", off[0]);
    for (int32_t g = 0; g < G; ++g)
        if (off[g + 1] < off[g]) return record_error(KMIP_ERR_INVALID_ARG, "graph_offsets decrease at %d", g);
    if (off[G] != N) return record_error(KMIP_ERR_INVALID_ARG, "graph_offsets[G]=%d != N=%lld", off[G], (long long)N);
    return KMIP_OK;
}

int32_t num_tiles(int64_t N) { return (int32_t)((N + 31) / 32); }

size_t packed_k_bytes(int64_t N, int32_t H, int32_t d) {
    return (size_t)H * (size_t)(num_tiles(N) + kmip::kPadTiles) * 32 * (size_t)d * 2;
}

// The tiled keys, before the counters.
size_t tiled_bytes(int64_t N, int32_t H, int32_t d) { return align_up(packed_k_bytes(N, H, d)); }

// The select kernel's per-XCD work counters and pacers, after the tiled keys.
constexpr size_t kCounterBytes = kmip::kSelectCounterBytes;

// Upper bound on the work-list length for any query-block size.
size_t max_tasks(int64_t N, int32_t G) { return (size_t)(N / 32 + G + 1); }

// Query blocks of 32 per wave: two when k and d are small and there are
// enough items to fill the chip, one otherwise (bounded by LDS per workgroup
// and, at d = 128, by registers).
// Candidate slots per lane: few, since LDS bounds the resident waves per CU
// and occupancy pays more than the extra merges cost (4 with two blocks, 8
// with one, measured on the 100k/500k/262k-node workloads).
kmip::SelectShape choose_shape(int64_t N, int32_t H, int32_t d, int32_t k, int32_t G) {
    const int64_t items = (N + 63) / 64 * H;
    if (k <= 32 && d <= 64 && items >= 8192 && G == 1) return kmip::SelectShape{2, 4};
    return kmip::SelectShape{1, 8};
}

// Queries are grouped by direction (group.hip) and keys stored in bounded
// superblocks (keyorder.hip) for a single graph large enough for the
// pre-passes to pay off, at d <= 64 (the key-order kernels are built for
// those widths).
bool use_grouping(int64_t N, int32_t G, int32_t d) { return G == 1 && N >= 8192 && d <= 64; }

// The small-graph select keeps up to KMIP_MAX_K_WIDE candidates per query
// in LDS and is built for d <= 64; other tasks go to the streaming kernel.
bool small_select_ok(int32_t d, int32_t k) { return d <= 64 && k <= KMIP_MAX_K_WIDE; }

// Workspace of kmip_topk_prefilter, in order: the bf16 key tiles and the
// select kernel's counters (for the query blocks it redoes), the int8 key
// tiles, the per-head quantisation figures, the candidate lists and their
// lengths, the overflow flags, the redo count and the redo task list.
struct PrefilterLayout {
    size_t tiles8, hstat, cand, ccount, flags, count, tasks, total;
};

PrefilterLayout prefilter_layout(int64_t N, int32_t H, int32_t d) {
    PrefilterLayout L{};
    const size_t nblocks = (size_t)num_tiles(N);
    size_t off = tiled_bytes(N, H, d) + kCounterBytes;
    L.tiles8 = off;
    off += align_up(kmip::prefilter_tile_bytes((int32_t)N, H, d));
    L.hstat = off;
    off += align_up((size_t)4 * H * sizeof(uint32_t));
    L.cand = off;
    off += align_up((size_t)N * H * kmip::kPrefilterCap * sizeof(int32_t));
    L.ccount = off;
    off += align_up((size_t)N * H * 2 * sizeof(int32_t));
    L.flags = off;
    off += align_up((size_t)H * nblocks * sizeof(int32_t));
    L.count = off;
    off += align_up(sizeof(int32_t));
    L.tasks = off;
    off += align_up(nblocks * sizeof(kmip::Task));
    L.total = off;
    return L;
}

// kmip_attend_ex with an optional query order (perm [H][N], the forward's
// grouping, or nullptr) for the order the aggregate takes query-heads in.
kmip_status_t attend_checked(const void* Q, const void* K, const void* V, int64_t N, int32_t H, int32_t d,
                             int32_t dv, int32_t k, float scale, const int32_t* topk_idx, const uint8_t* keep,
                             float drop_rate, const int32_t* perm, float* out, float* lse, void* stream_) {
    kmip_status_t s = check_sizes(N, H, d, k);
    if (s != KMIP_OK) return s;
    if ((s = check_value_width(N, H, dv)) != KMIP_OK) return s;
    if ((s = check_scale(scale)) != KMIP_OK) return s;
    if ((s = check_dropout(keep, drop_rate)) != KMIP_OK) return s;
    if (N == 0) return ok();
    if (!Q || !K || !V || !topk_idx || !out || !lse)
        return record_error(KMIP_ERR_INVALID_ARG, "null buffer passed to kmip_attend");
    if (!aligned16(Q) || !aligned16(K) || !aligned16(V))
        return record_error(KMIP_ERR_INVALID_ARG, "Q, K and V must be 16-byte aligned");
    hipError_t e = kmip::launch_attend(Q, K, V, topk_idx, keep, 1.0f / (1.0f - drop_rate), (int32_t)N, H, d, dv,
                                       k, scale, perm, out, lse, reinterpret_cast<hipStream_t>(stream_));
    if (e != hipSuccess) return hip_fail(e, "attend launch");
    return ok();
}

}  // namespace

extern "C" {

const char* kmip_status_string(kmip_status_t s) {
    switch (s) {
        case KMIP_OK: return "ok";
        case KMIP_ERR_INVALID_ARG: return "invalid argument";
        case KMIP_ERR_UNSUPPORTED: return "unsupported size";
        case KMIP_ERR_WORKSPACE: return "workspace missing or too small";
        case KMIP_ERR_HIP: return "HIP error";
    }
    return "unknown status";
}

const char* kmip_last_error(void) { return g_last_error.c_str(); }

size_t kmip_topk_workspace_size(int64_t N, int32_t H, int32_t d, int32_t k, int32_t num_graphs) {
    if (check_sizes(N, H, d, k) != KMIP_OK) return 0;
    const int32_t G = num_graphs < 1 ? 1 : num_graphs;
    size_t bytes = tiled_bytes(N, H, d) + kCounterBytes;
    if (G > 1) bytes += align_up(max_tasks(N, G) * sizeof(kmip::Task));
    if (use_grouping(N, G, d))
        bytes += align_up(kmip::group_workspace_bytes((int32_t)N, H, d)) +
                 align_up(kmip::key_order_workspace_bytes((int32_t)N, H, d));
    return bytes;
}

size_t kmip_fwd_workspace_size(int64_t N, int32_t H, int32_t d, int32_t k, int32_t num_graphs) {
    return kmip_topk_workspace_size(N, H, d, k, num_graphs);
}

kmip_status_t kmip_topk(const void* Q, const void* K, const int32_t* graph_offsets,
                        int32_t num_graphs, int64_t N, int32_t H, int32_t d, int32_t k,
                        int32_t* topk_idx, void* workspace, size_t workspace_bytes,
                        void* stream) {
    return kmip_topk_with_events(Q, K, graph_offsets, num_graphs, N, H, d, k, topk_idx, workspace,
                                 workspace_bytes, stream, nullptr, nullptr);
}

kmip_status_t kmip_topk_with_events(const void* Q, const void* K, const int32_t* graph_offsets,
                                    int32_t num_graphs, int64_t N, int32_t H, int32_t d, int32_t k,
                                    int32_t* topk_idx, void* workspace, size_t workspace_bytes,
                                    void* stream_, void* select_start, void* select_stop) {
    kmip_status_t s = check_sizes(N, H, d, k);
    if (s != KMIP_OK) return s;
    if ((s = check_offsets(graph_offsets, num_graphs, N)) != KMIP_OK) return s;
    if (N == 0) return ok();
    if (!Q || !K || !topk_idx) return record_error(KMIP_ERR_INVALID_ARG, "null Q, K or topk_idx");
    if (!aligned16(Q) || !aligned16(K)) return record_error(KMIP_ERR_INVALID_ARG, "Q and K must be 16-byte aligned");
    const int32_t G = graph_offsets ? num_graphs : 1;
    const size_t need = kmip_topk_workspace_size(N, H, d, k, G);
    if (workspace == nullptr || workspace_bytes < need)
        return record_error(KMIP_ERR_WORKSPACE, "workspace of %zu bytes < %zu required", workspace_bytes, need);
    if ((reinterpret_cast<uintptr_t>(workspace) & (kAlign - 1)) != 0)
        return record_error(KMIP_ERR_WORKSPACE, "workspace must be 256-byte aligned");
    hipStream_t stream = reinterpret_cast<hipStream_t>(stream_);

    const int32_t n32 = (int32_t)N;
    const int32_t ntiles = num_tiles(N);
    char* ws = reinterpret_cast<char*>(workspace);
    void* kp = ws;
    const kmip::SelectShape shape = choose_shape(N, H, d, k, G);
    const int32_t qb = shape.qb;

    const kmip::Task* dtasks = nullptr;
    int32_t ntasks = 0, nsmall = 0;
    if (G > 1) {
        // Block-diagonal batch: one task per run of 32*qb queries of a graph,
        // heaviest first (cost ~ queries x keys) to balance the tail.  The
        // tasks of graphs of at most kSmallGraph nodes (runs of 32 queries)
        // come first and go to the small-graph select (for the sizes it
        // takes).
        std::vector<kmip::Task> tasks;
        tasks.reserve(max_tasks(N, G));
        for (int pass = 0; pass < 2; ++pass) {
            const size_t first = tasks.size();
            for (int32_t g = 0; g < G; ++g) {
                const int32_t lo = graph_offsets[g], hi = graph_offsets[g + 1];
                const bool small = hi - lo <= kmip::kSmallGraph && small_select_ok(d, k);
                if (small != (pass == 0)) continue;
                const int32_t step = small ? 32 : 32 * qb;
                for (int32_t q0 = lo; q0 < hi; q0 += step)
                    tasks.push_back(kmip::Task{q0, std::min(step, hi - q0), lo, hi});
            }
            std::stable_sort(tasks.begin() + first, tasks.end(), [](const kmip::Task& a, const kmip::Task& b) {
                return (int64_t)a.q_count * (a.key_hi - a.key_lo) > (int64_t)b.q_count * (b.key_hi - b.key_lo);
            });
            if (pass == 0) nsmall = (int32_t)tasks.size();
        }
        ntasks = (int32_t)tasks.size() - nsmall;
        void* dst = ws + tiled_bytes(N, H, d) + kCounterBytes;
        hipError_t e = upload_async(dst, tasks.data(), tasks.size() * sizeof(kmip::Task), stream);
        if (e != hipSuccess) return hip_fail(e, "work list upload");
        dtasks = reinterpret_cast<const kmip::Task*>(dst) + nsmall;
    } else {
        ntasks = (int32_t)((N + 32 * qb - 1) / (32 * qb));
    }

    // A single large graph: queries grouped by direction, keys stored in
    // superblock order with bounds.
    kmip::QueryGroups groups{};
    kmip::KeyOrder keys{};
    const bool grouped = use_grouping(N, G, d);
    if (grouped) {
        char* gws = ws + tiled_bytes(N, H, d) + kCounterBytes;
        hipError_t e = kmip::launch_group_queries(Q, n32, H, d, gws, &groups, stream);
        if (e != hipSuccess) return hip_fail(e, "query grouping launch");
        char* kws = gws + align_up(kmip::group_workspace_bytes(n32, H, d));
        e = kmip::launch_key_order(K, n32, H, d, ntiles, kws, &keys, stream);
        if (e != hipSuccess) return hip_fail(e, "key order launch");
    }
    hipError_t e = kmip::launch_pack_k(K, grouped ? keys.perm : nullptr, grouped ? keys.rows : nullptr, kp, n32, H, d, ntiles,
                                          stream);
    if (e != hipSuccess) return hip_fail(e, "pack_k launch");
    int32_t* work_ctr = reinterpret_cast<int32_t*>(ws + tiled_bytes(N, H, d));
    hipEvent_t ev_start = reinterpret_cast<hipEvent_t>(select_start);
    hipEvent_t ev_stop = reinterpret_cast<hipEvent_t>(select_stop);
    if (nsmall > 0) {
        // the events bracket both select launches
        if (ev_start != nullptr && (e = hipEventRecord(ev_start, stream)) != hipSuccess)
            return hip_fail(e, "event record");
        ev_start = nullptr;
        e = kmip::launch_small_select(kp, Q, dtasks - nsmall, nsmall, n32, H, d, k, ntiles, topk_idx, stream);
        if (e != hipSuccess) return hip_fail(e, "small-graph select launch");
    }
    if (ntasks > 0) {
        e = kmip::launch_select(kp, Q, K, dtasks, grouped ? &groups : nullptr, grouped ? &keys : nullptr,
                                ntasks, n32, H, d, k, ntiles, shape, work_ctr, topk_idx, stream, ev_start, ev_stop);
        if (e != hipSuccess) return hip_fail(e, "select launch");
    } else if (ev_stop != nullptr && (e = hipEventRecord(ev_stop, stream)) != hipSuccess) {
        return hip_fail(e, "event record");
    }
    return ok();
}


size_t kmip_topk_prefilter_workspace_size(int64_t N, int32_t H, int32_t d, int32_t k) {
    if (check_sizes(N, H, d, k) != KMIP_OK || k > kmip::kPrefilterMaxK) return 0;
    return prefilter_layout(N, H, d).total;
}

kmip_status_t kmip_topk_prefilter(const void* Q, const void* K, int64_t N, int32_t H, int32_t d, int32_t k,
                                  int32_t* topk_idx, int32_t* redone, void* workspace, size_t workspace_bytes,
                                  void* stream_) {
    kmip_status_t s = check_sizes(N, H, d, k);
    if (s != KMIP_OK) return s;
    if (k > kmip::kPrefilterMaxK)
        return record_error(KMIP_ERR_UNSUPPORTED, "the prefilter takes k <= %d (got %d)", kmip::kPrefilterMaxK, k);
    if (N == 0) {
        hipError_t e = redone != nullptr ? kmip::launch_fill_zero(reinterpret_cast<float*>(redone), 1,
                                                                 reinterpret_cast<hipStream_t>(stream_))
                                         : hipSuccess;
        return e == hipSuccess ? ok() : hip_fail(e, "redo count");
    }
    if (!Q || !K || !topk_idx) return record_error(KMIP_ERR_INVALID_ARG, "null Q, K or topk_idx");
    if (!aligned16(Q) || !aligned16(K)) return record_error(KMIP_ERR_INVALID_ARG, "Q and K must be 16-byte aligned");
    const PrefilterLayout L = prefilter_layout(N, H, d);
    if (workspace == nullptr || workspace_bytes < L.total)
        return record_error(KMIP_ERR_WORKSPACE, "workspace of %zu bytes < %zu required", workspace_bytes, L.total);
    if ((reinterpret_cast<uintptr_t>(workspace) & (kAlign - 1)) != 0)
        return record_error(KMIP_ERR_WORKSPACE, "workspace must be 256-byte aligned");
    hipStream_t stream = reinterpret_cast<hipStream_t>(stream_);
    char* ws = reinterpret_cast<char*>(workspace);
    const int32_t n32 = (int32_t)N, ntiles = num_tiles(N);
    kmip::Task* tasks = reinterpret_cast<kmip::Task*>(ws + L.tasks);
    hipError_t e = kmip::launch_prefilter(K, Q, n32, H, d, k, reinterpret_cast<uint32_t*>(ws + L.hstat),
                                          reinterpret_cast<uint4*>(ws + L.tiles8), reinterpret_cast<int32_t*>(ws + L.cand),
                                          reinterpret_cast<int32_t*>(ws + L.ccount),
                                          reinterpret_cast<int32_t*>(ws + L.flags),
                                          reinterpret_cast<int32_t*>(ws + L.count), tasks, topk_idx, stream);
    if (e != hipSuccess) return hip_fail(e, "prefilter launch");
    // the query blocks whose candidate lists overflowed, through the select
    // kernel (every other entry of the list is a zero-query task it skips)
    if ((e = kmip::launch_pack_k(K, nullptr, nullptr, ws, n32, H, d, ntiles, stream)) != hipSuccess)
        return hip_fail(e, "pack_k launch");
    int32_t* work_ctr = reinterpret_cast<int32_t*>(ws + tiled_bytes(N, H, d));
    e = kmip::launch_select(ws, Q, K, tasks, nullptr, nullptr, ntiles, n32, H, d, k, ntiles, kmip::SelectShape{1, 8},
                            work_ctr, topk_idx, stream, nullptr, nullptr);
    if (e != hipSuccess) return hip_fail(e, "select launch");
    if (redone != nullptr &&
        (e = hipMemcpyAsync(redone, ws + L.count, sizeof(int32_t), hipMemcpyDeviceToDevice, stream)) != hipSuccess)
        return hip_fail(e, "redo count copy");
    return ok();
}

kmip_status_t kmip_attend_ex(const void* Q, const void* K, const void* V, int64_t N, int32_t H,
                             int32_t d, int32_t dv, int32_t k, float scale, const int32_t* topk_idx,
                             const uint8_t* keep, float drop_rate, float* out, float* lse, void* stream_) {
    return attend_checked(Q, K, V, N, H, d, dv, k, scale, topk_idx, keep, drop_rate, nullptr, out, lse, stream_);
}

kmip_status_t kmip_attend(const void* Q, const void* K, const void* V, int64_t N, int32_t H,
                          int32_t d, int32_t k, float scale, const int32_t* topk_idx, float* out,
                          float* lse, void* stream) {
    return kmip_attend_ex(Q, K, V, N, H, d, d, k, scale, topk_idx, nullptr, 0.0f, out, lse, stream);
}

kmip_status_t kmip_fwd_ex(const void* Q, const void* K, const void* V, const int32_t* graph_offsets,
                          int32_t num_graphs, int64_t N, int32_t H, int32_t d, int32_t dv, int32_t k,
                          float scale, const uint8_t* keep, float drop_rate, float* out, int32_t* topk_idx,
                          float* lse, void* workspace, size_t workspace_bytes, void* stream) {
    return kmip_fwd_ex_with_events(Q, K, V, graph_offsets, num_graphs, N, H, d, dv, k, scale, keep, drop_rate, out,
                                   topk_idx, lse, workspace, workspace_bytes, stream, nullptr, nullptr, nullptr);
}

kmip_status_t kmip_fwd_ex_with_events(const void* Q, const void* K, const void* V, const int32_t* graph_offsets,
                                      int32_t num_graphs, int64_t N, int32_t H, int32_t d, int32_t dv, int32_t k,
                                      float scale, const uint8_t* keep, float drop_rate, float* out,
                                      int32_t* topk_idx, float* lse, void* workspace, size_t workspace_bytes,
                                      void* stream, void* select_start, void* select_stop, void* attend_start) {
    kmip_status_t s = check_sizes(N, H, d, k);
    if (s != KMIP_OK) return s;
    if ((s = check_value_width(N, H, dv)) != KMIP_OK) return s;
    if ((s = check_scale(scale)) != KMIP_OK) return s;
    if ((s = check_dropout(keep, drop_rate)) != KMIP_OK) return s;
    if (N > 0 && (!V || !out || !lse)) return record_error(KMIP_ERR_INVALID_ARG, "null V, out or lse");
    if (N > 0 && !aligned16(V)) return record_error(KMIP_ERR_INVALID_ARG, "V must be 16-byte aligned");
    s = kmip_topk_with_events(Q, K, graph_offsets, num_graphs, N, H, d, k, topk_idx, workspace,
                              workspace_bytes, stream, select_start, select_stop);
    if (s != KMIP_OK) return s;
    if (N > 0 && attend_start != nullptr) {
        const hipError_t e = hipEventRecord(reinterpret_cast<hipEvent_t>(attend_start),
                                            reinterpret_cast<hipStream_t>(stream));
        if (e != hipSuccess) return hip_fail(e, "event record");
    }
    // one graph grouped by direction: the aggregate takes the queries in
    // that order too (the grouping is still in the workspace)
    const int32_t G = graph_offsets ? num_graphs : 1;
    const int32_t* perm = nullptr;
    if (N > 0 && use_grouping(N, G, d))
        perm = kmip::group_perm_in(reinterpret_cast<char*>(workspace) + tiled_bytes(N, H, d) + kCounterBytes,
                                   (int32_t)N, H, d);
    return attend_checked(Q, K, V, N, H, d, dv, k, scale, topk_idx, keep, drop_rate, perm, out, lse, stream);
}

kmip_status_t kmip_fwd(const void* Q, const void* K, const void* V, const int32_t* graph_offsets,
                       int32_t num_graphs, int64_t N, int32_t H, int32_t d, int32_t k,
                       float scale, float* out, int32_t* topk_idx, float* lse, void* workspace,
                       size_t workspace_bytes, void* stream) {
    return kmip_fwd_ex(Q, K, V, graph_offsets, num_graphs, N, H, d, d, k, scale, nullptr, 0.0f, out, topk_idx,
                       lse, workspace, workspace_bytes, stream);
}

// Backward variant the library picks (KMIP_BWD_AUTO): the bucketed reduction
// where the key rows fit its bucket table, the sizes are its own and the
// value width equals the key width, else the full key sort.
static int32_t default_bwd_variant(int64_t N, int32_t H, int32_t d, int32_t dv, int32_t k) {
    return dv == d && kmip::bwd_bucket_supported((int32_t)N, H, d, k) ? KMIP_BWD_BUCKETED : KMIP_BWD_SEGMENTED;
}

size_t kmip_bwd_ex_workspace_size(int64_t N, int32_t H, int32_t d, int32_t dv, int32_t k, int32_t variant) {
    if (check_sizes(N, H, d, k) != KMIP_OK || check_value_width(N, H, dv) != KMIP_OK) return 0;
    const int32_t v = variant == KMIP_BWD_AUTO ? default_bwd_variant(N, H, d, dv, k) : variant;
    if (v == KMIP_BWD_KEY_AGGREGATED) return align_up(kmip::bwd_agg_workspace_bytes((int32_t)N, H, d));
    if (v == KMIP_BWD_SEGMENTED) return align_up(kmip::bwd_csr_workspace_bytes((int32_t)N, H, k));
    if (v == KMIP_BWD_BUCKETED) return dv == d && kmip::bwd_bucket_supported((int32_t)N, H, d, k)
                                         ? align_up(kmip::bwd_bucket_workspace_bytes((int32_t)N, H, d, k))
                                         : 0;
    return 0;
}

size_t kmip_bwd_workspace_size(int64_t N, int32_t H, int32_t d, int32_t k, int32_t variant) {
    return kmip_bwd_ex_workspace_size(N, H, d, d, k, variant);
}

kmip_status_t kmip_bwd_ex(const void* Q, const void* K, const void* V, const void* dOut,
                          const int32_t* topk_idx, const float* lse, const uint8_t* keep, float drop_rate,
                          int64_t N, int32_t H, int32_t d, int32_t dv, int32_t k, float scale, float* dQ,
                          float* dK, float* dV, int32_t variant, void* workspace, size_t workspace_bytes,
                          void* stream_) {
    kmip_status_t s = check_sizes(N, H, d, k);
    if (s != KMIP_OK) return s;
    if ((s = check_value_width(N, H, dv)) != KMIP_OK) return s;
    if ((s = check_scale(scale)) != KMIP_OK) return s;
    if ((s = check_dropout(keep, drop_rate)) != KMIP_OK) return s;
    const float keep_scale = 1.0f / (1.0f - drop_rate);
    if (variant < KMIP_BWD_AUTO || variant > KMIP_BWD_KEY_AGGREGATED)
        return record_error(KMIP_ERR_UNSUPPORTED, "backward variant %d", variant);
    if (variant == KMIP_BWD_BUCKETED && dv != d)
        return record_error(KMIP_ERR_UNSUPPORTED, "the bucketed variant needs d_V == d_K (got %d, %d)", dv, d);
    if (N == 0) return ok();
    if (!Q || !K || !V || !dOut || !topk_idx || !lse || !dQ || !dK || !dV)
        return record_error(KMIP_ERR_INVALID_ARG, "null buffer passed to kmip_bwd");
    if (!aligned16(Q) || !aligned16(K) || !aligned16(V) || !aligned16(dOut))
        return record_error(KMIP_ERR_INVALID_ARG, "Q, K, V and dOut must be 16-byte aligned");
    if (!aligned16(dK) || !aligned16(dV)) return record_error(KMIP_ERR_INVALID_ARG, "dK and dV must be 16-byte aligned");
    const int32_t v = variant == KMIP_BWD_AUTO ? default_bwd_variant(N, H, d, dv, k) : variant;
    hipStream_t stream = reinterpret_cast<hipStream_t>(stream_);
    hipError_t e;
    if (v != KMIP_BWD_ATOMIC) {
        const size_t need = kmip_bwd_ex_workspace_size(N, H, d, dv, k, v);
        if (workspace == nullptr || workspace_bytes < need)
            return record_error(KMIP_ERR_WORKSPACE, "workspace of %zu bytes < %zu required", workspace_bytes, need);
        if ((reinterpret_cast<uintptr_t>(workspace) & (kAlign - 1)) != 0)
            return record_error(KMIP_ERR_WORKSPACE, "workspace must be 256-byte aligned");
    }
    if (v == KMIP_BWD_KEY_AGGREGATED) {
        e = kmip::launch_bwd_agg(Q, K, V, dOut, topk_idx, lse, keep, keep_scale, (int32_t)N, H, d, dv, k, scale,
                                 dQ, dK, dV, workspace, stream);
    } else if (v == KMIP_BWD_BUCKETED) {
        if (!kmip::bwd_bucket_supported((int32_t)N, H, d, k))
            return record_error(KMIP_ERR_UNSUPPORTED,
                                "the bucketed variant needs d <= 64, k <= 128 and N*H <= 8192*512 (key-row "
                                "buckets of at most 512 rows)");
        e = kmip::launch_bwd_bucket(Q, K, V, dOut, topk_idx, lse, keep, keep_scale, (int32_t)N, H, d, k, scale,
                                    dQ, dK, dV, workspace, stream);
    } else if (v == KMIP_BWD_SEGMENTED) {
        e = kmip::launch_bwd_csr(Q, K, V, dOut, topk_idx, lse, keep, keep_scale, (int32_t)N, H, d, dv, k, scale,
                                 dQ, dK, dV, workspace, stream);
    } else {
        e = kmip::launch_bwd_atomic(Q, K, V, dOut, topk_idx, lse, keep, keep_scale, (int32_t)N, H, d, dv, k,
                                    scale, dQ, dK, dV, stream);
    }
    if (e != hipSuccess) return hip_fail(e, "backward launch");
    return ok();
}

kmip_status_t kmip_bwd(const void* Q, const void* K, const void* V, const void* dOut,
                       const int32_t* topk_idx, const float* lse, int64_t N, int32_t H,
                       int32_t d, int32_t k, float scale, float* dQ, float* dK, float* dV,
                       int32_t variant, void* workspace, size_t workspace_bytes, void* stream) {
    return kmip_bwd_ex(Q, K, V, dOut, topk_idx, lse, nullptr, 0.0f, N, H, d, d, k, scale, dQ, dK, dV, variant,
                       workspace, workspace_bytes, stream);
}

}  // extern "C"
