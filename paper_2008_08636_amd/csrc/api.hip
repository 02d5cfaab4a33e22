// api.hip -- the C ABI declared in include/pardnn.h: argument checks, handle
// and memory management, launch sequencing. Every step runs in the kernels of
// structure.hip, levelize.hip, sweep.hip, sweep_pair.hip, critpath.hip,
// labelmem.hip, heuristics.hip, slicing.hip, clusters.hip and spanwork.hip
// (and the device sorts and scans they call); this file only checks,
// allocates and enqueues.
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <new>
#include <string>

#include <rocprofiler-sdk-roctx/roctx.h>

#include "internal.h"

using namespace pardnn;

// The batch workspace of pardnn_evaluate_batch_fixed, for callers that cannot
// allocate device memory. Each GPU the library runs on holds one copy until
// the process ends; every call on that GPU shares it and it keeps the last
// call's contents (nothing in it has to start at zero: each call writes what
// it reads). Host code reaches it only through the per-device address from
// hipGetSymbolAddress, never through the name.
static constexpr size_t kFixedScratchBytes = size_t(128) << 20;
static __device__ __align__(256) unsigned char scratch[kFixedScratchBytes];

namespace {

thread_local std::string g_last_error;

int hip_status(hipError_t e) {
    return e == hipErrorOutOfMemory || e == hipErrorMemoryAllocation ? PARDNN_E_NOMEM
                                                                     : PARDNN_E_DEVICE;
}

// Allocation-failure injection, for tests of the out-of-memory paths: with
// PARDNN_FAULT_ALLOC=n (n >= 1) in the environment, the n-th allocation the
// library attempts -- host or device, counted from the first attempt that
// sees this value of the variable -- fails as if memory were exhausted; later
// attempts succeed again. Unset, empty or n <= 0: no failures.
bool injected_alloc_failure() {
    static std::mutex m;
    static std::string seen;
    static long long count = 0;
    const char *e = std::getenv("PARDNN_FAULT_ALLOC");
    std::lock_guard<std::mutex> lock(m);
    if (e == nullptr || e[0] == 0) {
        seen.clear();
        count = 0;
        return false;
    }
    if (seen != e) {
        seen = e;
        count = 0;
    }
    const long long n = std::strtoll(e, nullptr, 10);
    return n > 0 && ++count == n;
}

// Every device allocation of the library goes through here (and the hook).
// On failure *p is null.
hipError_t dev_malloc(void **p, size_t bytes) {
    *p = nullptr;
    if (injected_alloc_failure()) return hipErrorOutOfMemory;
    const hipError_t e = hipMalloc(p, bytes);
    if (e != hipSuccess) *p = nullptr;
    return e;
}

#define HIP_TRY(expr)                                                                      \
    do {                                                                                   \
        hipError_t e_ = (expr);                                                            \
        if (e_ != hipSuccess)                                                              \
            return fail(hip_status(e_), std::string(#expr) + ": " + hipGetErrorString(e_)); \
    } while (0)

// Makes the handle's device current for the duration of a call and restores
// the caller's device afterwards.
struct DeviceScope {
    int prev = -1;
    bool ok = true;
    explicit DeviceScope(int dev) {
        if (hipGetDevice(&prev) != hipSuccess) {
            ok = false;
            return;
        }
        if (prev != dev && hipSetDevice(dev) != hipSuccess) ok = false;
    }
    ~DeviceScope() {
        int cur = -1;
        if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
    }
};

// A per-graph array, freed with the handle. Each such array has one size for
// the life of the handle, so one that an earlier, failed call already
// allocated is kept: a call that fails half-way (out of memory) leaves the
// handle fit for the next call, which allocates only what is missing.
template <class T>
hipError_t dalloc(Graph &g, T **p, size_t n) {
    if (*p != nullptr) return hipSuccess;
    if (n == 0) n = 1;
    void *q = nullptr;
    hipError_t e = dev_malloc(&q, n * sizeof(T));
    if (e != hipSuccess) return e;
    g.allocs.push_back(q);
    *p = static_cast<T *>(q);
    return hipSuccess;
}

void release(Graph *g) {
    (void)hipStreamSynchronize(g->stream);
    for (void *p : g->allocs) (void)hipFree(p);
    g->allocs.clear();
    if (g->batch_ws) (void)hipFree(g->batch_ws);
    if (g->aux_scratch) (void)hipFree(g->aux_scratch);
    if (g->h_err) (void)hipHostFree(g->h_err);
    if (g->ev0) (void)hipEventDestroy(g->ev0);
    if (g->ev1) (void)hipEventDestroy(g->ev1);
    delete g;
}

// Error words on the device: err[0] holds the argument-error flags that
// calls check on the device (bit meanings per call), err[1] the internal
// check of the secondary slicing walk.
//
// Start of a call that checks arguments on the device: clear the flags,
// unless errors are deferred (they then accumulate until taken).
hipError_t clear_errors(Graph *g) {
    if (g->defer_errors) return hipSuccess;
    return launch_fill_i32(g->err, 1, 0, g->stream);
}

// End of such a call: wait for the stream and copy the error words to the
// host. With errors deferred, no wait: the host copy reads as clear.
int read_errors(Graph *g) {
    if (g->defer_errors) {
        for (int i = 0; i < 4; i++) g->h_err[i] = 0;
        return PARDNN_OK;
    }
    HIP_TRY(hipMemcpyAsync(g->h_err, g->err, 4 * sizeof(int32_t), hipMemcpyDeviceToHost,
                           g->stream));
    HIP_TRY(hipStreamSynchronize(g->stream));
    return PARDNN_OK;
}

// Around the main kernels of a call (instrumentation only): a roctx range
// named for them, which a profiler's marker trace shows with the dispatches
// enqueued inside it, and, with timing on, an event pair on the stream.
struct TimedLaunch {
    Graph *g;
    TimedLaunch(Graph *g_, const char *name) : g(g_) {
        roctxRangePushA(name);
        if (g->timing) {
            g->timed_kernel = name;
            (void)hipEventRecord(g->ev0, g->stream);
        }
    }
    ~TimedLaunch() {
        if (g->timing) {
            (void)hipEventRecord(g->ev1, g->stream);
            g->timed = true;
        }
        roctxRangePop();
    }
};

int ensure_pair(Graph *g);

int ensure_levelized(Graph *g) {
    if (g->levelized) return PARDNN_OK;
    const int32_t V = g->V;
    HIP_TRY(dalloc(*g, &g->level, V));
    HIP_TRY(dalloc(*g, &g->order, V));
    HIP_TRY(dalloc(*g, &g->rank, (size_t)V + 1));   // rank[V] = -1: "no node"
    HIP_TRY(dalloc(*g, &g->level_ptr, (size_t)V + 2));
    // scratch: in-degree counters, the release queue, the result words, then
    // the level sort's own space
    const size_t sort_bytes = std::max(level_order_scratch_bytes(V), kahn_rec_bytes(V));
    const size_t head = (((size_t)V + 1) * 2 * sizeof(int32_t) + 8 + 255) / 256 * 256;
    char *work = nullptr;
    auto cleanup = [&]() {
        (void)hipStreamSynchronize(g->stream);
        if (work) (void)hipFree(work);
    };
    hipError_t e = dev_malloc((void **)&work, head + sort_bytes);
    int32_t *indeg_work = reinterpret_cast<int32_t *>(work);
    int32_t *queue = indeg_work + (V + 1);
    int32_t *result = queue + (V + 1);
    if (e == hipSuccess && V > 0)
        e = hipMemcpyAsync(indeg_work, g->indeg, sizeof(int32_t) * (size_t)V,
                           hipMemcpyDeviceToDevice, g->stream);
    if (e == hipSuccess) {
        TimedLaunch t(g, "k_kahn");
        e = launch_kahn(*g, indeg_work, queue, result, work + head);
    }
    int32_t h_result[2] = {0, 0};
    if (e == hipSuccess)
        e = hipMemcpyAsync(h_result, result, sizeof(h_result), hipMemcpyDeviceToHost, g->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(g->stream);
    if (e == hipSuccess && h_result[1] == V) {
        int32_t bits = 1;
        while (bits < 31 && (h_result[0] >> bits) != 0) bits++;
        e = launch_level_order(*g, bits, work + head);
    }
    cleanup();
    if (e != hipSuccess) return fail(hip_status(e), std::string("levelize: ") + hipGetErrorString(e));
    if (h_result[1] != V)
        return fail(PARDNN_E_CYCLE, "levelize: " + std::to_string(V - h_result[1]) +
                                        " node(s) lie on or behind a cycle");
    const int32_t L = h_result[0];
    g->L = L;
    g->h_level_ptr.assign((size_t)L + 1, 0);
    HIP_TRY(hipMemcpyAsync(g->h_level_ptr.data(), g->level_ptr, sizeof(int32_t) * ((size_t)L + 1),
                           hipMemcpyDeviceToHost, g->stream));
    HIP_TRY(hipStreamSynchronize(g->stream));
    int32_t mw = 0;
    for (int32_t k = 0; k < L; k++) mw = std::max(mw, g->h_level_ptr[k + 1] - g->h_level_ptr[k]);
    g->max_width = mw;

    const size_t E = (size_t)g->E;
    HIP_TRY(dalloc(*g, &g->linfo, (size_t)L + 2));
    HIP_TRY(dalloc(*g, &g->in_off, (size_t)V + 1));
    HIP_TRY(dalloc(*g, &g->in_src, E));
    HIP_TRY(dalloc(*g, &g->in_dst, E));
    HIP_TRY(dalloc(*g, &g->in_cost, E));
    HIP_TRY(dalloc(*g, &g->out_off, (size_t)V + 1));
    HIP_TRY(dalloc(*g, &g->out_src, E));
    HIP_TRY(dalloc(*g, &g->out_dst, E));
    HIP_TRY(dalloc(*g, &g->out_dst_orig, E));
    HIP_TRY(dalloc(*g, &g->out_cost, E));
    HIP_TRY(dalloc(*g, &g->comp_lm, V));
    HIP_TRY(dalloc(*g, &g->mem_lm, V));
    HIP_TRY(dalloc(*g, &g->in_rec, E));
    HIP_TRY(dalloc(*g, &g->out_rec, E));
    HIP_TRY(dalloc(*g, &g->node_rec, V));
    HIP_TRY(dalloc(*g, &g->lab_lm, V));
    HIP_TRY(dalloc(*g, &g->next_lm, V));
    HIP_TRY(dalloc(*g, &g->cp_flag, (size_t)V + 1));
    HIP_TRY(dalloc(*g, &g->cp_pos, (size_t)V + 1));
    HIP_TRY(dalloc(*g, &g->cp_ws, scan_workspace_elems(V)));
    HIP_TRY(dalloc(*g, &g->cp_list, V));
    HIP_TRY(dalloc(*g, &g->cp_ok, 1));
    HIP_TRY(dalloc(*g, &g->crit_lm, V));
    HIP_TRY(dalloc(*g, &g->ft_lm, 2 * (size_t)V));
    HIP_TRY(dalloc(*g, &g->bl_lm, 2 * (size_t)V));
    if (!g->move_stamp) {
        HIP_TRY(dalloc(*g, &g->move_stamp, V));
        HIP_TRY(launch_fill_i32(g->move_stamp, V, -1, g->stream));
    }

    int32_t *tmp = nullptr;
    const size_t scan_n = scan_workspace_elems(V);
    e = dev_malloc((void **)&tmp, sizeof(int32_t) * (4 * (size_t)V + scan_n + 4));
    if (e == hipSuccess)
        e = launch_build_lm(*g, tmp, tmp + 2 * (size_t)V, tmp + 3 * (size_t)V,
                            tmp + 4 * (size_t)V);
    if (e == hipSuccess) e = hipStreamSynchronize(g->stream);
    if (tmp) {
        (void)hipStreamSynchronize(g->stream);
        (void)hipFree(tmp);
    }
    if (e != hipSuccess) return fail(hip_status(e), std::string("levelize: ") + hipGetErrorString(e));
    // everything the batched evaluation needs besides its workspace is built
    // here, once per graph: the near / far edge split and the label-fit flag
    if (V > 0) {
        int st = ensure_pair(g);
        if (st != PARDNN_OK) return st;
    }
    HIP_TRY(dalloc(*g, &g->bt_fit, 1));
    g->levelized = true;
    return PARDNN_OK;
}

// Near / far edge split of the batched sweeps, built once per graph.
int ensure_pair(Graph *g) {
    if (g->pl_t != nullptr) return PARDNN_OK;
    const size_t E = (size_t)g->E;
    int32_t *flag = nullptr, *rank = nullptr, *ws = nullptr;
    auto cleanup = [&]() {
        (void)hipStreamSynchronize(g->stream);
        if (flag) (void)hipFree(flag);
        if (rank) (void)hipFree(rank);
        if (ws) (void)hipFree(ws);
    };
    hipError_t e = dev_malloc((void **)&flag, sizeof(int32_t) * (E + 1));
    if (e == hipSuccess) e = dev_malloc((void **)&rank, sizeof(int32_t) * (E + 1));
    if (e == hipSuccess)
        e = dev_malloc((void **)&ws, sizeof(int32_t) * scan_workspace_elems((int32_t)E));
    PairLevel *pl[2] = {nullptr, nullptr};
    NearRec12 *nr[2] = {nullptr, nullptr};
    FarRec16 *fr[2] = {nullptr, nullptr};
    for (int d = 0; d < 2 && e == hipSuccess; d++) {
        const bool fwd = d == 0;
        e = launch_fill_i32(rank, (int64_t)E + 1, 0, g->stream);
        if (e == hipSuccess && E > 0) e = launch_pair_flags(*g, fwd, flag);
        if (e == hipSuccess && E > 0)
            e = launch_exclusive_scan(flag, rank, (int32_t)E, ws, g->stream);
        int32_t n_near = 0;
        if (e == hipSuccess)
            e = hipMemcpyAsync(&n_near, rank + E, sizeof(int32_t), hipMemcpyDeviceToHost,
                               g->stream);
        if (e == hipSuccess) e = hipStreamSynchronize(g->stream);
        if (e == hipSuccess) e = dalloc(*g, &pl[d], (size_t)g->L + 2);
        if (e == hipSuccess) e = dalloc(*g, &nr[d], (size_t)n_near);
        if (e == hipSuccess) e = dalloc(*g, &fr[d], E - (size_t)n_near);
        if (e == hipSuccess)
            e = launch_pair_split(*g, fwd, rank, pl[d], nr[d], fr[d]);
        int32_t *&lsrc = fwd ? g->lsrc_t : g->lsrc_b;
        if (e == hipSuccess) e = dalloc(*g, &lsrc, (size_t)long_list_elems(g->L));
        if (e == hipSuccess) e = launch_long_blocks(*g, fwd, pl[d], fr[d], lsrc);
        // edges that wide levels fold early
        if (e == hipSuccess) e = hipStreamSynchronize(g->stream);
        if (e == hipSuccess) e = launch_fill_i32(rank, (int64_t)E + 1, 0, g->stream);
        if (e == hipSuccess && E > 0) e = launch_pre_flags(*g, fwd, flag);
        if (e == hipSuccess && E > 0)
            e = launch_exclusive_scan(flag, rank, (int32_t)E, ws, g->stream);
        int32_t n_pre = 0;
        if (e == hipSuccess)
            e = hipMemcpyAsync(&n_pre, rank + E, sizeof(int32_t), hipMemcpyDeviceToHost,
                               g->stream);
        if (e == hipSuccess) e = hipStreamSynchronize(g->stream);
        int32_t *&preoff = fwd ? g->preoff_t : g->preoff_b;
        PreRec16 *&pre = fwd ? g->pre_t : g->pre_b;
        if (e == hipSuccess) e = dalloc(*g, &preoff, (size_t)g->L + 1);
        if (e == hipSuccess) e = dalloc(*g, &pre, (size_t)n_pre);
        if (e == hipSuccess && !fwd) e = dalloc(*g, &g->pretie_b, (size_t)n_pre);
        if (e == hipSuccess)
            e = launch_pre_split(*g, fwd, rank, preoff, pre, fwd ? nullptr : g->pretie_b);
    }
    cleanup();
    if (e != hipSuccess) return fail(hip_status(e), std::string("batch structure: ") + hipGetErrorString(e));
    g->pl_t = pl[0];
    g->pl_b = pl[1];
    g->nr_t = nr[0];
    g->nr_b = nr[1];
    g->fr_t = fr[0];
    g->fr_b = fr[1];
    return PARDNN_OK;
}

SweepArgs sweep_args(const Graph *g) {
    SweepArgs a{};
    a.V = g->V;
    a.E = g->E;
    a.L = g->L;
    a.linfo = g->linfo;
    a.in_off = g->in_off;
    a.in_src = g->in_src;
    a.in_dst = g->in_dst;
    a.in_cost = g->in_cost;
    a.out_off = g->out_off;
    a.out_src = g->out_src;
    a.out_dst = g->out_dst;
    a.out_dst_orig = g->out_dst_orig;
    a.out_cost = g->out_cost;
    a.comp_lm = g->comp_lm;
    a.mem_lm = g->mem_lm;
    a.in_rec = g->in_rec;
    a.out_rec = g->out_rec;
    a.node_rec = g->node_rec;
    a.order = g->order;
    a.lab_stride = g->V;
    a.level = g->level;
    a.level_ptr = g->level_ptr;
    a.rank = g->rank;
    a.err = g->err;
    return a;
}

#define CHECK_HANDLE(g)                                            \
    do {                                                           \
        if ((g) == nullptr) return fail(PARDNN_E_INVAL, "null handle"); \
    } while (0)

#define DEVICE_SCOPE(g)                                                         \
    DeviceScope scope_((g)->device);                                            \
    if (!scope_.ok) return fail(PARDNN_E_DEVICE, "cannot select the handle's device")

// Placements come either as a [V][P] matrix or as base + per-step moves.
struct MovesIn {
    const int32_t *base;
    const int64_t *step_ptr;
    int64_t n_moves;   // host value: the length of node and label
    const int32_t *node, *label;
};

// With `fixed` the batch workspace is the caller-provided block of
// fixed_bytes (no allocation on this path); the handle must then already be
// levelized.
int evaluate_impl(Graph *g, int32_t n_place, const int32_t *placements, const MovesIn *mv,
                  int32_t n_labels, const int64_t *capacity, int64_t *tl, int64_t *bl,
                  int64_t *makespan, uint8_t *is_critical, int32_t *path, int32_t path_stride,
                  int32_t *path_len, int64_t *label_mem, int64_t *overflow,
                  void *fixed = nullptr, size_t fixed_bytes = 0) {
    if (n_place < 0) return fail(PARDNN_E_INVAL, "n_place must be >= 0");
    if (n_place == 0) return PARDNN_OK;
    if (makespan == nullptr || (g->V > 0 && placements == nullptr && mv == nullptr))
        return fail(PARDNN_E_INVAL, "placements and makespan must be non-null");
    if ((path == nullptr) != (path_len == nullptr))
        return fail(PARDNN_E_INVAL, "path and path_len must both be given or both be null");
    if (label_mem == nullptr && overflow != nullptr)
        return fail(PARDNN_E_INVAL, "overflow needs label_mem");
    if (label_mem != nullptr && n_labels < 1) return fail(PARDNN_E_INVAL, "n_labels must be >= 1");
    DEVICE_SCOPE(g);
    if (fixed != nullptr && !g->levelized)
        return fail(PARDNN_E_INVAL, "the graph must be levelized (pardnn_levelize) before a "
                                    "call that allocates nothing");
    int st = ensure_levelized(g);
    if (st != PARDNN_OK) return st;
    if (path != nullptr && path_stride < std::max(g->L, 1))
        return fail(PARDNN_E_INVAL, "path_stride must be at least the number of levels");

    const int32_t S = kBatchSlots;
    const int64_t n_slices = (n_place + S - 1) / S;
    // ftl, bll, nx_w: per slice (V + kSlicePad) x S elements (room for
    // stores of idle lanes); lab_w: V x S per slice. Both strides are rounded
    // up to 256 bytes, so that every slice starts on a cache line and a run
    // of nodes touches no more lines than its size needs.
    const int64_t ws_stride = (((int64_t)g->V + kSlicePad) * S + 31) / 32 * 32;
    const int64_t lab_stride = ((int64_t)g->V * S + 63) / 64 * 64;
    const size_t per = (size_t)n_slices * (size_t)ws_stride;
    const size_t per_lab = (size_t)n_slices * (size_t)lab_stride;
    // The pair sweep reads 16-bit labels (a node's two labels of a slice are
    // one 4-byte word): half the bytes for the label build to write and for
    // the sweep to read. They have a region of their own, lab_h, so that a
    // call without label sums can keep 32-bit labels in lab_w for its
    // unpacked alternative.
    const int64_t lab_elems16 = ((int64_t)g->V * S + 127) / 128 * 128;
    const size_t lab_h_bytes = ((size_t)n_slices * (size_t)lab_elems16 * 2 + 255) / 256 * 256;
    // successive placements from moves: the number of moves sizes the scratch
    // that groups them by node
    int64_t n_moves = 0;
    if (mv != nullptr) {
        if (mv->n_moves < 0 || mv->n_moves >= (int64_t)INT32_MAX)
            return fail(PARDNN_E_INVAL, "n_moves must lie in [0, 2^31)");
        if (mv->n_moves > 0 && (mv->node == nullptr || mv->label == nullptr))
            return fail(PARDNN_E_INVAL, "node and label must be non-null");
        if (g->V > 0 && mv->base == nullptr) return fail(PARDNN_E_INVAL, "base must be non-null");
        n_moves = mv->n_moves;   // step_ptr is checked against it on the device
    }
    const size_t moves_bytes =
        mv != nullptr ? (moves_scratch_elems(g->V, n_moves) * sizeof(int32_t) + 255) / 256 * 256
                      : 0;
    // critical bit words for the path walk: [P][ceil(V / 32)]
    const size_t cbits_bytes =
        path != nullptr ? (((size_t)g->V + 31) / 32 * (size_t)n_place * 4 + 255) / 256 * 256 : 0;
    // ftl, bll: room for 16-byte pairs; lab_w, nx_w: int32; start: [P]; the
    // 16-bit labels; then the critical bit words and the moves scratch
    const size_t need = per * (4 * sizeof(int64_t) + sizeof(int32_t)) +
                        per_lab * sizeof(int32_t) + (size_t)n_place * sizeof(int32_t) + 1024 +
                        lab_h_bytes + cbits_bytes + moves_bytes;
    void *ws_base = nullptr;
    if (fixed != nullptr) {
        if (need > fixed_bytes)
            return fail(PARDNN_E_INVAL,
                        "the batch needs " + std::to_string(need) + " bytes of workspace; the "
                        "fixed workspace holds " + std::to_string(fixed_bytes) +
                        " (fewer placements per call fit)");
        ws_base = fixed;
    } else {
        if (g->batch_ws_bytes < need) {
            if (g->batch_ws) {
                HIP_TRY(hipStreamSynchronize(g->stream));
                HIP_TRY(hipFree(g->batch_ws));
                g->batch_ws = nullptr;
                g->batch_ws_bytes = 0;
            }
            HIP_TRY(dev_malloc(&g->batch_ws, need));
            g->batch_ws_bytes = need;
        }
        ws_base = g->batch_ws;
    }
    // Pack {value, label} into one int64 when labels are known to lie in
    // [0, n_labels) (they are checked) and values leave room for their bits.
    // The b keys then also carry the successor id: (value << ob) | (2^ob - 1 - id)
    // with 2^ob > V, which needs values below 2^(62 - ob) as well.
    // Without label sums the labels are unchecked: those below 2^16 -- or
    // below n_labels, when the caller gives it as a hint in [1, 2^16], which
    // leaves fewer label bits and room for the successor links -- still fit,
    // which the label build finds out on the device (bt_fit); then both sweeps
    // are enqueued and the one that does not apply returns at once, so the
    // call needs no host round trip to choose.
    int32_t lb = 0, ob = 0;
    bool gated = false;
    const int64_t label_range = label_mem != nullptr ? (int64_t)n_labels
                                : n_labels >= 1 && (uint32_t)n_labels <= kPackLabels
                                    ? (int64_t)n_labels
                                    : (int64_t)kPackLabels;
    if (g->V > 0) {
        int32_t bits = 1;
        while ((1ll << bits) < label_range) bits++;
        const int32_t obits = succ_bits(g->V);
        const int32_t wide = std::max(bits, obits);
        if (bits <= 16 && wide < 62 && g->weight_bound < (1ll << (62 - wide))) {
            lb = bits;
            ob = obits;
            gated = label_mem == nullptr;
        }
    }

    int64_t *ftl = (int64_t *)ws_base;
    int64_t *bll = ftl + 2 * per;
    int32_t *lab_w = (int32_t *)(bll + 2 * per);
    int32_t *nx_w = lab_w + per_lab;
    int32_t *start = nx_w + per;
    // after start[P], on a 256-byte boundary
    const size_t lab_h_off = (per * (4 * sizeof(int64_t) + sizeof(int32_t)) +
                              per_lab * sizeof(int32_t) + (size_t)n_place * sizeof(int32_t) + 255) /
                             256 * 256;
    int32_t *lab_h = reinterpret_cast<int32_t *>((char *)ws_base + lab_h_off);
    uint32_t *cbits = reinterpret_cast<uint32_t *>(
        (char *)ws_base + (need - moves_bytes - cbits_bytes) / 256 * 256);
    int32_t *moves_scratch = reinterpret_cast<int32_t *>(
        (char *)ws_base + (need - moves_bytes) / 256 * 256);

    const int32_t K = label_mem != nullptr ? n_labels : 0;
    int32_t *fit = gated ? g->bt_fit : nullptr;
    // The labels the pair sweep reads are 16-bit: checked at their full width
    // (against K, or for a call without label sums against 2^lb, which sets
    // the fit flag) as the workspace is built. A call without label sums then
    // writes the 32-bit labels for its unpacked alternative only when some
    // label does not fit: that pass reads the fit flag on the device and
    // returns at once otherwise.
    const bool lab16 = lb > 0 && g->V > 0;
    int32_t *lab_sweep = lab16 ? lab_h : lab_w;
    const int64_t lab_elems = lab16 ? lab_elems16 : lab_stride;
    HIP_TRY(clear_errors(g));
    if (fit != nullptr) HIP_TRY(launch_fill_i32(fit, 1, 1, g->stream));
    if (mv != nullptr) {
        HIP_TRY(launch_check_steps(mv->step_ptr, n_place, n_moves, g->err, g->stream));
        HIP_TRY(launch_moves_to_slices(*g, mv->base, n_place, mv->step_ptr, n_moves, mv->node,
                                       mv->label, S, moves_scratch, lab_sweep, lab_elems, K,
                                       g->err, fit, 1u << lb, lab16));
        if (gated)
            HIP_TRY(launch_moves_write(*g, mv->base, n_place, n_moves, S, moves_scratch, lab_w,
                                       lab_stride, fit, 0));
    } else {
        HIP_TRY(launch_permute_labels_batch(*g, placements, n_place, S, lab_sweep, lab_elems, K,
                                            g->err, fit, 1u << lb, lab16));
        if (gated)
            HIP_TRY(launch_permute_labels_batch(*g, placements, n_place, S, lab_w, lab_stride, 0,
                                                nullptr, nullptr, kPackLabels, false, fit, 0));
    }
    if (K > 0) {
        HIP_TRY(launch_fill_i64(label_mem, (int64_t)n_place * K, 0, g->stream));
    }
    SweepArgs a = sweep_args(g);
    a.P = n_place;
    a.K = K;
    a.lab_w = lab_sweep;
    a.lab_stride = lab_elems;
    a.lab16 = lab16 ? 1 : 0;
    a.ftl = ftl;
    a.bll = bll;
    a.nx_w = path != nullptr ? nx_w : nullptr;
    a.tl_out = tl;
    a.bl_out = bl;
    a.makespan = makespan;
    a.start = path != nullptr ? start : nullptr;
    a.label_mem = label_mem;
    a.lb = lb;
    a.ob = ob;
    a.ws_stride = ws_stride;
    if (lb > 0 && g->V > 0) {
        a.pl_t = g->pl_t;
        a.pl_b = g->pl_b;
        a.nr_t = g->nr_t;
        a.nr_b = g->nr_b;
        a.fr_t = g->fr_t;
        a.fr_b = g->fr_b;
        a.lsrc_t = g->lsrc_t;
        a.lsrc_b = g->lsrc_b;
        a.preoff_t = g->preoff_t;
        a.preoff_b = g->preoff_b;
        a.pre_t = g->pre_t;
        a.pre_b = g->pre_b;
        a.pretie_b = g->pretie_b;
    }
    // The successor links ride in the packed b values when those have room
    // for them (a gated call's unpacked alternative writes nx_w instead; the
    // path walk reads the gate to know which)
    a.nxf = path != nullptr && lb > 0 && lb + ob < 62 &&
                    g->weight_bound < (1ll << (62 - lb - ob))
                ? 1
                : 0;
    // the unpacked alternative of a gated call: {value, label} pairs
    SweepArgs alt = a;
    alt.lb = 0;
    alt.ob = 0;
    alt.nxf = 0;
    alt.lab_w = lab_w;   // the 32-bit labels of the gated second pass
    alt.lab_stride = lab_stride;
    alt.lab16 = 0;
    alt.gate = fit;
    alt.gate_want = 0;
    if (gated) {
        a.gate = fit;
        a.gate_want = 1;
    }
    if (lb > 0 && g->V > 0) {
        TimedLaunch t(g, gated ? "k_sweep_pair<2> or k_sweep<2>" : "k_sweep_pair<2>");
        HIP_TRY(launch_sweep_pair(a, g->stream));
        if (gated) HIP_TRY(launch_sweep(alt, S, g->stream));
    } else {
        TimedLaunch t(g, "k_sweep<2>");
        HIP_TRY(launch_sweep(a, S, g->stream));
    }
    HIP_TRY(launch_finish(a, S, is_critical, cbits, path, path_stride, path_len, g->stream,
                          gated ? &alt : nullptr));
    if (K > 0) {
        if (overflow != nullptr || capacity != nullptr)
            HIP_TRY(launch_overflow((int64_t)n_place * K, K, capacity, label_mem, overflow, g->err,
                                    g->stream));
    }
    if (K > 0 || mv != nullptr) {
        st = read_errors(g);
        if (st != PARDNN_OK) return st;
        if (g->h_err[0] & 1)
            return fail(PARDNN_E_INVAL, mv != nullptr && K == 0
                                            ? "a moved node id is outside [0, n_nodes)"
                                            : "a label or a moved node id is out of range");
        if (g->h_err[0] & 2) return fail(PARDNN_E_INVAL, "a capacity is negative");
        if (g->h_err[0] & kErrSteps)
            return fail(PARDNN_E_INVAL, "step_ptr must start at 0, never decrease and end at "
                                        "n_moves");
    }
    return PARDNN_OK;
}


// One placement through the batched pair sweep, for the single-placement
// passes of slicing and cluster criticality: the pair kernel's per-level chain
// is shorter than the single sweep's. Its packed keys hold labels below 2^lb
// (lb <= 16) and values of magnitude up to `bound`; pair_single_bits says
// whether they fit and sets lb / ob.
bool pair_single_bits(const Graph *g, int64_t n_labels, int64_t bound, int32_t *lb,
                      int32_t *ob) {
    int32_t bits = 1;
    while ((1ll << bits) < n_labels) bits++;
    const int32_t obits = succ_bits(g->V);
    const int32_t wide = std::max(bits, obits);
    if (bits > 16 || wide >= 62 || bound >= (1ll << (62 - wide))) return false;
    *lb = bits;
    *ob = obits;
    return true;
}

// one placement per chain: workspace V + pad values, labels V
constexpr int64_t ps_ws_stride(int32_t V) { return ((int64_t)V + kSlicePad + 31) / 32 * 32; }
constexpr int64_t ps_lab_stride(int32_t V) { return ((int64_t)V + 63) / 64 * 64; }

// labels (original ids) into the pair sweep's level-major layout
int pair_single_labels(Graph *g, const int32_t *labels) {
    const int32_t V = g->V;
    HIP_TRY(dalloc(*g, &g->ps_ftl, (size_t)ps_ws_stride(V)));
    HIP_TRY(dalloc(*g, &g->ps_bll, (size_t)ps_ws_stride(V)));
    HIP_TRY(dalloc(*g, &g->ps_lab, (size_t)ps_lab_stride(V)));
    HIP_TRY(dalloc(*g, &g->ps_gate, 1));
    HIP_TRY(launch_permute_labels_batch(*g, labels, 1, 1, g->ps_lab, ps_lab_stride(V)));
    return PARDNN_OK;
}

// Levels wider than this many nodes are computed grid-wide between chain
// segments in single-placement sweeps (environment PARDNN_WIDE_LEVEL; 0 or
// less: never).
int32_t wide_level_threshold() {
    const char *e = std::getenv("PARDNN_WIDE_LEVEL");
    if (e != nullptr && e[0] != 0) return (int32_t)std::strtol(e, nullptr, 10);
    return 512;
}

// The plan of a segmented sweep for threshold `thr`: per direction, runs of
// chain steps and the wide levels between them (cached on the handle).
int seg_plan(Graph *g, int32_t thr) {
    if (g->seg_thresh == thr) return PARDNN_OK;
    if (g->h_linfo.empty()) {   // once per graph: the level bounds on the host
        g->h_linfo.resize((size_t)g->L + 2);
        HIP_TRY(hipMemcpyAsync(g->h_linfo.data(), g->linfo, sizeof(LevelInfo) * ((size_t)g->L + 2),
                               hipMemcpyDeviceToHost, g->stream));
        HIP_TRY(hipStreamSynchronize(g->stream));
    }
    g->seg_thresh = thr;
    g->seg_t.clear();
    g->seg_b.clear();
    const int32_t L = g->L;
    auto wide = [&](int32_t x) {
        return thr > 0 && g->h_level_ptr[x + 1] - g->h_level_ptr[x] > thr;
    };
    for (int d = 0; d < 2; d++) {
        std::vector<SegItem> &out = d == 0 ? g->seg_t : g->seg_b;
        int32_t start = 0;
        for (int32_t st = 0; st < L; st++) {
            const int32_t x = d == 0 ? st : L - 1 - st;
            if (!wide(x)) continue;
            if (st > start) out.push_back({0, start, st});
            out.push_back({1, x, 0});
            start = st + 1;
        }
        if (start < L) out.push_back({0, start, L});
    }
    return PARDNN_OK;
}

// tl, bl (original order) and the level-0 makespan of the labels set by
// pair_single_labels, with the given node weights; with `gate`, the launches
// run only if *gate == 1
int pair_single_sweep(Graph *g, int32_t lb, int32_t ob, NodeRec16 *node_rec, int64_t *comp_lm,
                      int64_t *tl, int64_t *bl, int64_t *makespan, const int32_t *gate = nullptr,
                      bool timed = true) {
    int st = ensure_pair(g);
    if (st != PARDNN_OK) return st;
    SweepArgs a = sweep_args(g);
    a.P = 1;
    a.K = 0;
    a.lab_w = g->ps_lab;
    a.lab_stride = ps_lab_stride(g->V);
    a.ftl = g->ps_ftl;
    a.bll = g->ps_bll;
    a.ws_stride = ps_ws_stride(g->V);
    a.nx_w = nullptr;
    a.start = nullptr;
    a.label_mem = nullptr;
    a.tl_out = tl;
    a.bl_out = bl;
    a.makespan = makespan;
    a.node_rec = node_rec;
    a.comp_lm = comp_lm;
    a.lb = lb;
    a.ob = ob;
    a.pl_t = g->pl_t;
    a.pl_b = g->pl_b;
    a.nr_t = g->nr_t;
    a.nr_b = g->nr_b;
    a.fr_t = g->fr_t;
    a.fr_b = g->fr_b;
    a.lsrc_t = g->lsrc_t;
    a.lsrc_b = g->lsrc_b;
    a.preoff_t = g->preoff_t;
    a.preoff_b = g->preoff_b;
    a.pre_t = g->pre_t;
    a.pre_b = g->pre_b;
    a.pretie_b = g->pretie_b;
    a.gate = gate;
    a.gate_want = 1;
    const int32_t thr = wide_level_threshold();
    const bool segmented = thr > 0 && g->max_width > thr;
    if (!segmented) {
        if (timed) {
            TimedLaunch t(g, "k_sweep_pair<1>");
            HIP_TRY(launch_sweep_pair_one(a, g->stream));
        } else {
            HIP_TRY(launch_sweep_pair_one(a, g->stream));
        }
    } else {
        // chain segments for the narrow runs, grid-wide passes for the wide
        // levels; the t and b plans advance one item per round, paired in the
        // same launches (the two directions are independent)
        st = seg_plan(g, thr);
        if (st != PARDNN_OK) return st;
        if (!g->ps_acc) {
            HIP_TRY(dalloc(*g, &g->ps_acc, 2 * (size_t)std::max(g->max_width, 1)));
            HIP_TRY(launch_fill_i64(reinterpret_cast<int64_t *>(g->ps_acc),
                                    2 * (int64_t)std::max(g->max_width, 1), 0, g->stream));
        }
        auto run = [&]() -> int {
        const size_t nt = g->seg_t.size(), nb = g->seg_b.size();
        for (size_t r = 0; r < std::max(nt, nb); r++) {
            const SegItem *it = r < nt ? &g->seg_t[r] : nullptr;
            const SegItem *ib = r < nb ? &g->seg_b[r] : nullptr;
            SweepArgs x = a;
            x.seg_on = 1;
            x.seg_t0 = x.seg_t1 = x.seg_b0 = x.seg_b1 = 0;
            if (it && it->kind == 0) {
                x.seg_t0 = it->a;
                x.seg_t1 = it->b;
            }
            if (ib && ib->kind == 0) {
                x.seg_b0 = ib->a;
                x.seg_b1 = ib->b;
            }
            if (x.seg_t1 > x.seg_t0 || x.seg_b1 > x.seg_b0)
                HIP_TRY(launch_sweep_pair_one(x, g->stream));
            const int32_t xt = it && it->kind == 1 ? it->a : -1;
            const int32_t xb = ib && ib->kind == 1 ? ib->a : -1;
            if (xt >= 0 || xb >= 0) {
                const auto &li = g->h_linfo;
                const int32_t wt = xt >= 0 ? li[xt + 1].node_lo - li[xt].node_lo : 0;
                const int32_t wb = xb >= 0 ? li[xb + 1].node_lo - li[xb].node_lo : 0;
                const int64_t et = xt >= 0 ? li[xt + 1].in_e_lo - li[xt].in_e_lo : 0;
                const int64_t eb = xb >= 0 ? li[xb + 1].out_e_lo - li[xb].out_e_lo : 0;
                HIP_TRY(launch_wide_level(a, xt, xb, et + eb, wt + wb, g->ps_acc,
                                          g->ps_acc + std::max(g->max_width, 1), g->stream));
            }
        }
        HIP_TRY(launch_level0_makespan(a, g->stream));
        return PARDNN_OK;
        };
        if (timed) {
            TimedLaunch t(g, "segmented k_sweep_pair<1> + k_wide_*");
            st = run();
        } else {
            st = run();
        }
        if (st != PARDNN_OK) return st;
    }
    HIP_TRY(launch_finish(a, 1, nullptr, nullptr, nullptr, 0, nullptr, g->stream));
    return PARDNN_OK;
}

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on device `dev`, which must be current; looked
// up once per device.
int fixed_scratch(int dev, void **out) {
    if (dev < 0 || dev >= kMaxDevices) return fail(PARDNN_E_DEVICE, "device index out of range");
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_ptr[dev] == nullptr) {
        void *ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress((void **)&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess || ptr == nullptr)
            return fail(PARDNN_E_DEVICE, std::string("hipGetSymbolAddress(scratch): ") +
                                             hipGetErrorString(e));
        g_scratch_ptr[dev] = ptr;
    }
    *out = g_scratch_ptr[dev];
    return PARDNN_OK;
}

}  // namespace

int pardnn::fail(int status, const std::string &msg) {
    g_last_error = msg;
    return status;
}

extern "C" {

const char *pardnn_status_string(int status) {
    switch (status) {
        case PARDNN_OK: return "ok";
        case PARDNN_E_INVAL: return "invalid argument";
        case PARDNN_E_CYCLE: return "graph has a cycle";
        case PARDNN_E_OVERFLOW: return "weights overflow int64";
        case PARDNN_E_NOMEM: return "device out of memory";
        case PARDNN_E_DEVICE: return "device or HIP runtime error";
        default: return "unknown status";
    }
}

const char *pardnn_last_error(void) { return g_last_error.c_str(); }

int pardnn_graph_create(int32_t n_nodes, int64_t n_edges, const int32_t *src, const int32_t *dst,
                        const int64_t *comp, const int64_t *edge_cost, const int64_t *mem,
                        void *stream, pardnn_graph **out) {
    g_last_error.clear();
    if (out == nullptr) return fail(PARDNN_E_INVAL, "out is null");
    *out = nullptr;
    if (n_nodes < 0 || n_nodes > PARDNN_MAX_NODES || n_edges < 0 || n_edges > PARDNN_MAX_EDGES)
        return fail(PARDNN_E_INVAL, "need 0 <= n_nodes <= 2^26 and 0 <= n_edges <= 2^27");
    if (n_edges > 0 && (src == nullptr || dst == nullptr || edge_cost == nullptr))
        return fail(PARDNN_E_INVAL, "src, dst and edge_cost must be non-null when n_edges > 0");
    if (n_nodes > 0 && (comp == nullptr || mem == nullptr))
        return fail(PARDNN_E_INVAL, "comp and mem must be non-null when n_nodes > 0");
    // the handle first: a host allocation, which needs no device
    Graph *g = injected_alloc_failure() ? nullptr : new (std::nothrow) Graph();
    if (g == nullptr) return fail(PARDNN_E_NOMEM, "host allocation of the handle failed");
    int ndev = 0;
    if (hipGetDeviceCount(&ndev) != hipSuccess || ndev <= 0) {
        delete g;
        return fail(PARDNN_E_DEVICE, "no HIP device available");
    }
    if (hipGetDevice(&g->device) != hipSuccess) {
        delete g;
        return fail(PARDNN_E_DEVICE, "hipGetDevice failed");
    }
    int lds = 0;
    if (hipDeviceGetAttribute(&lds, hipDeviceAttributeMaxSharedMemoryPerBlock, g->device) ==
            hipSuccess &&
        lds > 0)
        g->lds_max = (size_t)lds;
    g->stream = (hipStream_t)stream;
    g->V = n_nodes;
    g->E = n_edges;
    int st = [&]() -> int {
        const size_t V = (size_t)n_nodes, E = (size_t)n_edges;
        HIP_TRY(dalloc(*g, &g->e_src, E));
        HIP_TRY(dalloc(*g, &g->e_dst, E));
        HIP_TRY(dalloc(*g, &g->e_cost, E));
        HIP_TRY(dalloc(*g, &g->comp, V));
        HIP_TRY(dalloc(*g, &g->mem, V));
        HIP_TRY(dalloc(*g, &g->indeg, V));
        HIP_TRY(dalloc(*g, &g->outdeg, V));
        HIP_TRY(dalloc(*g, &g->o_off, V + 1));
        HIP_TRY(dalloc(*g, &g->o_nbr, E));
        HIP_TRY(dalloc(*g, &g->err, 4));
        if (injected_alloc_failure())
            return fail(PARDNN_E_NOMEM, "host allocation of the error words failed");
        HIP_TRY(hipHostMalloc((void **)&g->h_err, 4 * sizeof(int32_t), hipHostMallocDefault));
        ValidateAcc *acc = nullptr;
        HIP_TRY(dalloc(*g, &acc, 1));
        HIP_TRY(hipMemsetAsync(acc, 0, sizeof(ValidateAcc), g->stream));
        HIP_TRY(launch_validate(*g, src, dst, comp, edge_cost, mem, acc));
        ValidateAcc h{};
        HIP_TRY(hipMemcpyAsync(&h, acc, sizeof(h), hipMemcpyDeviceToHost, g->stream));
        HIP_TRY(hipStreamSynchronize(g->stream));
        if (h.flags & 1ull) return fail(PARDNN_E_INVAL, "an edge endpoint is outside [0, n_nodes)");
        if (h.flags & 2ull) return fail(PARDNN_E_INVAL, "a weight (comp, edge_cost or mem) is negative");
        const unsigned __int128 w = ((unsigned __int128)h.w_hi << 32) + h.w_lo;
        const unsigned __int128 m = ((unsigned __int128)h.m_hi << 32) + h.m_lo;
        if (w > (unsigned __int128)INT64_MAX)
            return fail(PARDNN_E_OVERFLOW, "sum(comp) + sum(edge_cost) exceeds INT64_MAX");
        if (m > (unsigned __int128)INT64_MAX)
            return fail(PARDNN_E_OVERFLOW, "sum(mem) exceeds INT64_MAX");
        g->weight_bound = (int64_t)w;
        if (E > 0) {
            HIP_TRY(hipMemcpyAsync(g->e_src, src, E * sizeof(int32_t), hipMemcpyDeviceToDevice, g->stream));
            HIP_TRY(hipMemcpyAsync(g->e_dst, dst, E * sizeof(int32_t), hipMemcpyDeviceToDevice, g->stream));
            HIP_TRY(hipMemcpyAsync(g->e_cost, edge_cost, E * sizeof(int64_t), hipMemcpyDeviceToDevice, g->stream));
        }
        if (V > 0) {
            HIP_TRY(hipMemcpyAsync(g->comp, comp, V * sizeof(int64_t), hipMemcpyDeviceToDevice, g->stream));
            HIP_TRY(hipMemcpyAsync(g->mem, mem, V * sizeof(int64_t), hipMemcpyDeviceToDevice, g->stream));
        }
        HIP_TRY(launch_fill_i32(g->indeg, (int64_t)V, 0, g->stream));
        HIP_TRY(launch_fill_i32(g->outdeg, (int64_t)V, 0, g->stream));
        HIP_TRY(launch_count_degrees(*g));
        int32_t *ws = nullptr;
        HIP_TRY(dev_malloc((void **)&ws, sizeof(int32_t) * (scan_workspace_elems(n_nodes) + V + 1)));
        hipError_t e = launch_exclusive_scan(g->outdeg, g->o_off, n_nodes, ws, g->stream);
        if (e == hipSuccess) e = launch_build_orig_csr(*g, ws + scan_workspace_elems(n_nodes));
        if (e == hipSuccess) e = hipStreamSynchronize(g->stream);
        (void)hipStreamSynchronize(g->stream);
        (void)hipFree(ws);
        HIP_TRY(e);
        return PARDNN_OK;
    }();
    if (st != PARDNN_OK) {
        std::string msg = g_last_error;
        release(g);
        g_last_error = msg;
        return st;
    }
    *out = reinterpret_cast<pardnn_graph *>(g);
    return PARDNN_OK;
}

int pardnn_graph_destroy(pardnn_graph *h) {
    if (h == nullptr) return PARDNN_OK;
    Graph *g = reinterpret_cast<Graph *>(h);
    DeviceScope scope(g->device);
    release(g);
    return PARDNN_OK;
}

int pardnn_set_stream(pardnn_graph *h, void *stream) {
    CHECK_HANDLE(h);
    reinterpret_cast<Graph *>(h)->stream = (hipStream_t)stream;
    return PARDNN_OK;
}

int pardnn_get_info(const pardnn_graph *h, pardnn_info *info) {
    CHECK_HANDLE(h);
    if (info == nullptr) return fail(PARDNN_E_INVAL, "info is null");
    const Graph *g = reinterpret_cast<const Graph *>(h);
    info->n_nodes = g->V;
    info->n_edges = g->E;
    info->n_levels = g->levelized ? g->L : -1;
    info->max_width = g->levelized ? g->max_width : -1;
    info->device = g->device;
    return PARDNN_OK;
}

int pardnn_levelize(pardnn_graph *h, int32_t *level, int32_t *order, int32_t *level_ptr,
                    int32_t *n_levels_host) {
    CHECK_HANDLE(h);
    Graph *g = reinterpret_cast<Graph *>(h);
    DEVICE_SCOPE(g);
    g_last_error.clear();
    int st = ensure_levelized(g);
    if (st != PARDNN_OK) return st;
    const size_t V = (size_t)g->V;
    if (level && V)
        HIP_TRY(hipMemcpyAsync(level, g->level, V * sizeof(int32_t), hipMemcpyDeviceToDevice, g->stream));
    if (order && V)
        HIP_TRY(hipMemcpyAsync(order, g->order, V * sizeof(int32_t), hipMemcpyDeviceToDevice, g->stream));
    if (level_ptr)
        HIP_TRY(hipMemcpyAsync(level_ptr, g->level_ptr, ((size_t)g->L + 1) * sizeof(int32_t),
                               hipMemcpyDeviceToDevice, g->stream));
    if (n_levels_host) *n_levels_host = g->L;
    return PARDNN_OK;
}

int pardnn_tb_levels(pardnn_graph *h, const int32_t *placement, int64_t *tl, int64_t *bl,
                     int64_t *makespan) {
    CHECK_HANDLE(h);
    Graph *g = reinterpret_cast<Graph *>(h);
    if (makespan == nullptr || (g->V > 0 && (placement == nullptr || tl == nullptr || bl == nullptr)))
        return fail(PARDNN_E_INVAL, "placement, tl, bl and makespan must be non-null");
    DEVICE_SCOPE(g);
    int st = ensure_levelized(g);
    if (st != PARDNN_OK) return st;
    // Labels below 2^16 fit the pair sweep's packed keys. Whether they do is
    // decided on the device: both paths are enqueued and the one that does
    // not apply returns at once, so the call stays asynchronous.
    int32_t lb = 0, ob = 0;
    const bool pair = g->V > 0 && pair_single_bits(g, 1 << 16, g->weight_bound, &lb, &ob);
    if (pair) {
        st = ensure_pair(g);
        if (st == PARDNN_OK) st = pair_single_labels(g, placement);
        if (st != PARDNN_OK) return st;
    }
    HIP_TRY(launch_permute_labels(*g, placement, g->lab_lm));
    SweepArgs a = sweep_args(g);
    a.P = 1;
    a.K = 0;
    a.lab_w = g->lab_lm;
    a.lab_stride = g->V;
    a.ftl = g->ft_lm;
    a.bll = g->bl_lm;
    a.ws_stride = g->V;
    a.tl_out = tl;
    a.bl_out = bl;
    a.makespan = makespan;
    TimedLaunch t(g, pair ? "k_sweep_pair<1> or k_sweep<1>" : "k_sweep<1>");
    if (pair) {
        HIP_TRY(launch_label_fit(*g, placement, 1 << 16, g->ps_gate));
        st = pair_single_sweep(g, lb, ob, g->node_rec, g->comp_lm, tl, bl, makespan, g->ps_gate,
                               false);
        if (st != PARDNN_OK) return st;
        a.gate = g->ps_gate;
        a.gate_want = 0;
    }
    HIP_TRY(launch_sweep(a, 1, g->stream));
    return PARDNN_OK;
}

int pardnn_critical_path(pardnn_graph *h, const int32_t *placement, const int64_t *tl,
                         const int64_t *bl, const int64_t *makespan, uint8_t *is_critical,
                         int32_t *path, int32_t *path_len) {
    CHECK_HANDLE(h);
    Graph *g = reinterpret_cast<Graph *>(h);
    if (makespan == nullptr || path_len == nullptr ||
        (g->V > 0 && (placement == nullptr || tl == nullptr || bl == nullptr ||
                      is_critical == nullptr || path == nullptr)))
        return fail(PARDNN_E_INVAL, "all arguments of pardnn_critical_path must be non-null");
    DEVICE_SCOPE(g);
    int st = ensure_levelized(g);
    if (st != PARDNN_OK) return st;
    HIP_TRY(launch_critical_path(*g, placement, tl, bl, makespan, is_critical, path, path_len));
    return PARDNN_OK;
}

int pardnn_label_memory(pardnn_graph *h, const int32_t *placement, int32_t n_labels,
                        const int64_t *capacity, int64_t *label_mem, int64_t *overflow) {
    CHECK_HANDLE(h);
    Graph *g = reinterpret_cast<Graph *>(h);
    if (n_labels < 1) return fail(PARDNN_E_INVAL, "n_labels must be >= 1");
    if (label_mem == nullptr || (g->V > 0 && placement == nullptr))
        return fail(PARDNN_E_INVAL, "placement and label_mem must be non-null");
    DEVICE_SCOPE(g);
    HIP_TRY(clear_errors(g));
    HIP_TRY(launch_label_memory(*g, placement, n_labels, capacity, label_mem, overflow, g->err));
    int st = read_errors(g);
    if (st != PARDNN_OK) return st;
    if (g->h_err[0] & 1) return fail(PARDNN_E_INVAL, "a label lies outside [0, n_labels)");
    if (g->h_err[0] & 2) return fail(PARDNN_E_INVAL, "a capacity is negative");
    return PARDNN_OK;
}

int pardnn_memory_balance(pardnn_graph *h, int32_t n_place, const int32_t *placements,
                          const int32_t *node_type, const int32_t *ref_target, int32_t n_labels,
                          int64_t *res_mem, int64_t *nor_mem, uint8_t *balanced,
                          int64_t *ref_misplaced) {
    CHECK_HANDLE(h);
    Graph *g = reinterpret_cast<Graph *>(h);
    if (n_place < 0) return fail(PARDNN_E_INVAL, "n_place must be >= 0");
    if (n_labels < 1) return fail(PARDNN_E_INVAL, "n_labels must be >= 1");
    if (n_place == 0) return PARDNN_OK;
    if (res_mem == nullptr || nor_mem == nullptr || balanced == nullptr || ref_misplaced == nullptr)
        return fail(PARDNN_E_INVAL, "res_mem, nor_mem, balanced and ref_misplaced must be non-null");
    if (g->V > 0 && (placements == nullptr || node_type == nullptr || ref_target == nullptr))
        return fail(PARDNN_E_INVAL, "placements, node_type and ref_target must be non-null");
    DEVICE_SCOPE(g);
    HIP_TRY(clear_errors(g));
    // the events bracket the sums kernel alone (recorded inside the launch)
    if (g->timing && g->V > 0) {
        g->timed_kernel = "k_mem_balance_sums";
        g->timed = true;
    }
    HIP_TRY(launch_mem_balance(*g, n_place, placements, node_type, ref_target, n_labels, res_mem,
                               nor_mem, balanced, ref_misplaced, g->err));
    int st = read_errors(g);
    if (st != PARDNN_OK) return st;
    if (g->h_err[0] & 1) return fail(PARDNN_E_INVAL, "a label lies outside [0, n_labels)");
    if (g->h_err[0] & 2) return fail(PARDNN_E_INVAL, "a node kind is not 0, 1 or 2");
    if (g->h_err[0] & 4) return fail(PARDNN_E_INVAL, "a reference target lies outside [-1, n_nodes)");
    return PARDNN_OK;
}

// Scratch of the cluster and span calls, grown on demand (calls on one handle
// are ordered on its stream; the old block is freed only after a sync).
hipError_t grow_aux(Graph *g, size_t need) {
    if (g->aux_scratch_bytes >= need) return hipSuccess;
    hipError_t e;
    if (g->aux_scratch) {
        if ((e = hipStreamSynchronize(g->stream)) != hipSuccess) return e;
        if ((e = hipFree(g->aux_scratch)) != hipSuccess) return e;
        g->aux_scratch = nullptr;
        g->aux_scratch_bytes = 0;
    }
    if ((e = dev_malloc(&g->aux_scratch, need)) != hipSuccess) return e;
    g->aux_scratch_bytes = need;
    return hipSuccess;
}

int pardnn_span_work(pardnn_graph *h, const int32_t *label, int32_t K, const int32_t *cluster,
                     int32_t n_clusters, const int64_t *tl, int64_t *span_lo, int64_t *span_hi,
                     int64_t *work, int64_t *comm, int32_t *choice) {
    CHECK_HANDLE(h);
    Graph *g = reinterpret_cast<Graph *>(h);
    if (K < 1) return fail(PARDNN_E_INVAL, "K must be >= 1");
    if (n_clusters < 0) return fail(PARDNN_E_INVAL, "n_clusters must be >= 0");
    if (g->V > 0 && (label == nullptr || cluster == nullptr || tl == nullptr))
        return fail(PARDNN_E_INVAL, "label, cluster and tl must be non-null");
    if (n_clusters > 0 && (span_lo == nullptr || span_hi == nullptr || work == nullptr ||
                           comm == nullptr || choice == nullptr))
        return fail(PARDNN_E_INVAL, "output pointers must be non-null");
    if (n_clusters == 0 && g->V == 0) return PARDNN_OK;
    DEVICE_SCOPE(g);
    int st = ensure_levelized(g);
    if (st != PARDNN_OK) return st;
    HIP_TRY(grow_aux(g, span_work_scratch_bytes(g->V, n_clusters, K)));
    if (g->span_cache.changed == nullptr) {
        HIP_TRY(dalloc(*g, &g->span_cache.tl, g->V));
        HIP_TRY(dalloc(*g, &g->span_cache.ids, g->V));
        HIP_TRY(dalloc(*g, &g->span_cache.changed, 1));
    }
    HIP_TRY(clear_errors(g));
    {
        TimedLaunch t(g, "span_work");
        HIP_TRY(launch_span_work(*g, label, K, cluster, n_clusters, tl, span_lo, span_hi, work,
                                 comm, choice, g->aux_scratch, &g->span_cache, g->err));
    }
    st = read_errors(g);
    if (st != PARDNN_OK) return st;
    if (g->h_err[0] & 1) return fail(PARDNN_E_INVAL, "a cluster id lies outside [-1, n_clusters)");
    if (g->h_err[0] & 2) return fail(PARDNN_E_INVAL, "a label lies outside [-1, K)");
    return PARDNN_OK;
}

int pardnn_cluster_criticality(pardnn_graph *h, const int32_t *cluster, int32_t n_clusters,
                               int64_t *criticality, int32_t *order) {
    CHECK_HANDLE(h);
    Graph *g = reinterpret_cast<Graph *>(h);
    if (n_clusters < 0 || (n_clusters == 0 && g->V > 0))
        return fail(PARDNN_E_INVAL, "n_clusters must be >= 1 (>= 0 for an empty graph)");
    if (n_clusters == 0) return PARDNN_OK;
    if (criticality == nullptr || order == nullptr || (g->V > 0 && cluster == nullptr))
        return fail(PARDNN_E_INVAL, "cluster, criticality and order must be non-null");
    DEVICE_SCOPE(g);
    int st = ensure_levelized(g);
    if (st != PARDNN_OK) return st;
    const int32_t V = g->V;
    if (V > 0 && !g->cl_m) {
        HIP_TRY(dalloc(*g, &g->cl_tl, V));
        HIP_TRY(dalloc(*g, &g->cl_bl, V));
        HIP_TRY(dalloc(*g, &g->cl_m, 1));
    }
    const size_t sort_bytes = (cluster_sort_bytes(V, n_clusters) + 255) / 256 * 256;
    HIP_TRY(grow_aux(g, sort_bytes + cluster_relabel_bytes(V, n_clusters)));
    HIP_TRY(clear_errors(g));
    // The pair sweep packs labels below 2^16. The cluster ids fit when there
    // are few clusters; otherwise labels with the same equality on every edge
    // (levels for lone nodes, L + rank for the others) often do.
    int32_t lb = 0, ob = 0;
    const int32_t *pair_labels = nullptr;
    if (V > 0) {
        int32_t *lab = nullptr, *n_multi = nullptr;
        HIP_TRY(launch_cluster_relabel(
            *g, cluster, n_clusters,
            reinterpret_cast<int32_t *>(reinterpret_cast<char *>(g->aux_scratch) + sort_bytes),
            &lab, &n_multi));
        int32_t h_multi = 0;
        HIP_TRY(hipMemcpyAsync(&h_multi, n_multi, sizeof(int32_t), hipMemcpyDeviceToHost,
                               g->stream));
        HIP_TRY(hipStreamSynchronize(g->stream));
        if (pair_single_bits(g, (int64_t)g->L + h_multi, g->weight_bound, &lb, &ob))
            pair_labels = lab;
        else if (pair_single_bits(g, n_clusters, g->weight_bound, &lb, &ob))
            pair_labels = cluster;
    }
    if (pair_labels != nullptr) {
        st = pair_single_labels(g, pair_labels);
        if (st == PARDNN_OK)
            st = pair_single_sweep(g, lb, ob, g->node_rec, g->comp_lm, g->cl_tl, g->cl_bl,
                                   g->cl_m);
        if (st != PARDNN_OK) return st;
    } else if (V > 0) {
        // weighted levels with the cluster ids as labels: communication inside
        // a cluster is zero
        HIP_TRY(launch_permute_labels(*g, cluster, g->lab_lm));
        SweepArgs a = sweep_args(g);
        a.P = 1;
        a.K = 0;
        a.lab_w = g->lab_lm;
        a.lab_stride = V;
        a.ftl = g->ft_lm;
        a.bll = g->bl_lm;
        a.ws_stride = V;
        a.tl_out = g->cl_tl;
        a.bl_out = g->cl_bl;
        a.makespan = g->cl_m;
        TimedLaunch t(g, "k_sweep<1>");
        HIP_TRY(launch_sweep(a, 1, g->stream));
    }
    HIP_TRY(launch_cluster_criticality(*g, cluster, n_clusters, g->cl_tl, g->cl_bl, criticality,
                                       order, g->aux_scratch, sort_bytes, g->err));
    st = read_errors(g);
    if (st != PARDNN_OK) return st;
    if (g->h_err[0] & 1) return fail(PARDNN_E_INVAL, "a cluster id lies outside [0, n_clusters)");
    return PARDNN_OK;
}

}  // extern "C"

namespace {

// The K rounds of Alg. 1 (slicing primaries) on a levelized graph with V > 0;
// with `then_levels`, one more evaluation of the graph that remains (its tl /
// bl in sl_tl / sl_bl), for the secondary clusters.
int slice_rounds(Graph *g, int32_t K, int32_t *primary, int32_t *paths, int32_t path_stride,
                 int32_t *path_len, int64_t *makespan, bool then_levels) {
    const int32_t V = g->V;
    if (!g->sl_m) {   // the last of the group (an earlier failed call may have made some)
        HIP_TRY(dalloc(*g, &g->sl_node_rec, V));
        HIP_TRY(dalloc(*g, &g->sl_comp, V));
        HIP_TRY(dalloc(*g, &g->sl_tl, V));
        HIP_TRY(dalloc(*g, &g->sl_bl, V));
        HIP_TRY(dalloc(*g, &g->sl_alive, V));
        HIP_TRY(dalloc(*g, &g->sl_crit, V));
        HIP_TRY(dalloc(*g, &g->sl_iota, V));
        HIP_TRY(dalloc(*g, &g->sl_start, 1));
        HIP_TRY(dalloc(*g, &g->sl_m, 1));
        // every node its own label: before placement all communication counts
        HIP_TRY(launch_iota_i32(g->sl_iota, V, g->stream));
    }
    // a removed node weighs -B with B above every path length
    const int64_t big = g->weight_bound < INT64_MAX ? g->weight_bound + 1 : INT64_MAX;
    HIP_TRY(launch_slice_init(*g, g->sl_node_rec, g->sl_comp, g->sl_alive, primary));
    // Every edge joins two levels, so the level as label makes every edge pay,
    // as distinct labels do: with fewer than 2^16 levels the rounds can take
    // the pair sweep (values lie in [-B, B]).
    int32_t lb = 0, ob = 0;
    const bool pair = (K > 0 || then_levels) && big < INT64_MAX &&
                      pair_single_bits(g, g->L, big, &lb, &ob);
    if (pair) {
        const int st = pair_single_labels(g, g->level);
        if (st != PARDNN_OK) return st;
    }
    auto sweep = [&](int64_t *m) -> int {
        if (pair)
            return pair_single_sweep(g, lb, ob, g->sl_node_rec, g->sl_comp, g->sl_tl, g->sl_bl, m);
        SweepArgs a = sweep_args(g);
        a.P = 1;
        a.K = 0;
        a.lab_w = g->order;   // pairwise distinct labels in level-major order
        a.lab_stride = V;
        a.ftl = g->ft_lm;
        a.bll = g->bl_lm;
        a.ws_stride = V;
        a.tl_out = g->sl_tl;
        a.bl_out = g->sl_bl;
        a.makespan = m;
        a.node_rec = g->sl_node_rec;
        a.comp_lm = g->sl_comp;
        TimedLaunch t(g, "k_sweep<1>");
        HIP_TRY(launch_sweep(a, 1, g->stream));
        return PARDNN_OK;
    };
    for (int32_t j = 0; j < K; j++) {
        int st = sweep(makespan + j);
        if (st != PARDNN_OK) return st;
        HIP_TRY(launch_slice_makespan(*g, g->sl_alive, g->sl_tl, g->sl_bl, makespan + j));
        HIP_TRY(launch_crit_next(*g, g->sl_iota, g->sl_comp, g->sl_tl, g->sl_bl, makespan + j,
                                 g->sl_crit));
        HIP_TRY(launch_slice_start(*g, g->sl_alive, g->sl_start));
        int32_t *pj = paths + (int64_t)j * path_stride;
        HIP_TRY(launch_chase_from(*g, g->sl_start, pj, path_len + j));
        HIP_TRY(launch_slice_remove(*g, j, pj, path_len + j, big, g->sl_node_rec, g->sl_comp,
                                    g->sl_alive, primary));
    }
    if (then_levels) return sweep(g->sl_m);
    return PARDNN_OK;
}

}  // namespace

extern "C" {

int pardnn_slice_primaries(pardnn_graph *h, int32_t K, int32_t *primary, int32_t *paths,
                           int32_t path_stride, int32_t *path_len, int64_t *makespan) {
    CHECK_HANDLE(h);
    Graph *g = reinterpret_cast<Graph *>(h);
    if (K < 0) return fail(PARDNN_E_INVAL, "K must be >= 0");
    if (K > 0 && (path_len == nullptr || makespan == nullptr || paths == nullptr))
        return fail(PARDNN_E_INVAL, "paths, path_len and makespan must be non-null");
    if (g->V > 0 && primary == nullptr) return fail(PARDNN_E_INVAL, "primary must be non-null");
    DEVICE_SCOPE(g);
    int st = ensure_levelized(g);
    if (st != PARDNN_OK) return st;
    if (K > 0 && path_stride < std::max(g->L, 1))
        return fail(PARDNN_E_INVAL, "path_stride must be at least the number of levels");
    if (g->V == 0) {
        if (K > 0) {
            HIP_TRY(launch_fill_i32(path_len, K, 0, g->stream));
            HIP_TRY(launch_fill_i64(makespan, K, 0, g->stream));
        }
        return PARDNN_OK;
    }
    return slice_rounds(g, K, primary, paths, path_stride, path_len, makespan, false);
}

int pardnn_slice_graph(pardnn_graph *h, int32_t K, int32_t *cluster, int32_t *cluster_off,
                       int32_t *cluster_nodes, int32_t *n_clusters, int64_t *makespan) {
    CHECK_HANDLE(h);
    Graph *g = reinterpret_cast<Graph *>(h);
    if (K < 0) return fail(PARDNN_E_INVAL, "K must be >= 0");
    if (cluster_off == nullptr || n_clusters == nullptr ||
        (g->V > 0 && (cluster == nullptr || cluster_nodes == nullptr)))
        return fail(PARDNN_E_INVAL, "cluster, cluster_off, cluster_nodes and n_clusters must "
                                    "be non-null");
    DEVICE_SCOPE(g);
    int st = ensure_levelized(g);
    if (st != PARDNN_OK) return st;
    const int32_t V = g->V;
    const int32_t stride = std::max(g->L, 1);
    // scratch: primary paths [K][stride], their lengths and makespans, then
    // the walk's own space
    const size_t paths_bytes = ((size_t)K * stride * 4 + 255) / 256 * 256;
    const size_t small_bytes = ((size_t)K * 12 + 255) / 256 * 256;
    HIP_TRY(grow_aux(g, paths_bytes + small_bytes + peel_scratch_bytes(V, g->E)));
    char *base = reinterpret_cast<char *>(g->aux_scratch);
    int32_t *paths = reinterpret_cast<int32_t *>(base);
    int64_t *ms = reinterpret_cast<int64_t *>(base + paths_bytes);
    int32_t *plen = reinterpret_cast<int32_t *>(ms + K);
    void *peel = base + paths_bytes + small_bytes;
    HIP_TRY(launch_fill_i32(g->err + 1, 1, 0, g->stream));
    if (V == 0) {
        HIP_TRY(launch_fill_i32(cluster_off, (int64_t)K + 1, 0, g->stream));
        HIP_TRY(launch_fill_i32(n_clusters, 1, K, g->stream));
        if (makespan != nullptr && K > 0) HIP_TRY(launch_fill_i64(makespan, K, 0, g->stream));
        return PARDNN_OK;
    }
    st = slice_rounds(g, K, cluster, paths, stride, plen, makespan != nullptr ? makespan : ms,
                      true);
    if (st != PARDNN_OK) return st;
    const char *env = std::getenv("PARDNN_PEEL_GLOBAL_MAPS");
    const bool force_global = env != nullptr && env[0] == '1';
    const bool lds = !force_global && peel_lds_bytes(V) <= g->lds_max;
    {
        TimedLaunch t(g, "secondary clusters");
        HIP_TRY(launch_slice_secondaries(*g, K, paths, stride, plen, g->sl_tl, g->sl_bl,
                                         g->sl_alive, cluster, cluster_off, cluster_nodes,
                                         n_clusters, peel, lds, g->err + 1));
    }
    // an internal check, never deferred
    int32_t walk_err = 0;
    HIP_TRY(hipMemcpyAsync(&walk_err, g->err + 1, sizeof(int32_t), hipMemcpyDeviceToHost,
                           g->stream));
    HIP_TRY(hipStreamSynchronize(g->stream));
    if (walk_err & 1) return fail(PARDNN_E_DEVICE, "the secondary walk stopped early");
    return PARDNN_OK;
}

int pardnn_apply_moves(pardnn_graph *h, int32_t *placement, int32_t n_moves, const int32_t *node,
                       const int32_t *label) {
    CHECK_HANDLE(h);
    Graph *g = reinterpret_cast<Graph *>(h);
    if (n_moves < 0) return fail(PARDNN_E_INVAL, "n_moves must be >= 0");
    if (n_moves == 0) return PARDNN_OK;
    if (placement == nullptr || node == nullptr || label == nullptr)
        return fail(PARDNN_E_INVAL, "placement, node and label must be non-null");
    DEVICE_SCOPE(g);
    if (!g->move_stamp) {
        HIP_TRY(dalloc(*g, &g->move_stamp, g->V));
        HIP_TRY(launch_fill_i32(g->move_stamp, g->V, -1, g->stream));
    }
    HIP_TRY(clear_errors(g));
    HIP_TRY(launch_apply_moves(*g, placement, n_moves, node, label, g->err));
    int st = read_errors(g);
    if (st != PARDNN_OK) return st;
    if (g->h_err[0] & 1) return fail(PARDNN_E_INVAL, "a moved node id is outside [0, n_nodes)");
    return PARDNN_OK;
}

int pardnn_build_placements(pardnn_graph *h, const int32_t *base, int32_t n_place,
                            const int64_t *step_ptr, int64_t n_moves, const int32_t *node,
                            const int32_t *label, int32_t *placements) {
    CHECK_HANDLE(h);
    Graph *g = reinterpret_cast<Graph *>(h);
    if (n_place < 0) return fail(PARDNN_E_INVAL, "n_place must be >= 0");
    if (n_place == 0) return PARDNN_OK;
    if (step_ptr == nullptr || (g->V > 0 && (base == nullptr || placements == nullptr)))
        return fail(PARDNN_E_INVAL, "base, step_ptr and placements must be non-null");
    if (n_moves < 0 || n_moves >= (int64_t)INT32_MAX)
        return fail(PARDNN_E_INVAL, "n_moves must lie in [0, 2^31)");
    if (n_moves > 0 && (node == nullptr || label == nullptr))
        return fail(PARDNN_E_INVAL, "node and label must be non-null");
    DEVICE_SCOPE(g);
    HIP_TRY(clear_errors(g));
    HIP_TRY(launch_check_steps(step_ptr, n_place, n_moves, g->err, g->stream));
    HIP_TRY(launch_build_placements(*g, base, n_place, step_ptr, n_moves, node, label, placements,
                                    g->err));
    int st = read_errors(g);
    if (st != PARDNN_OK) return st;
    if (g->h_err[0] & 1) return fail(PARDNN_E_INVAL, "a moved node id is outside [0, n_nodes)");
    if (g->h_err[0] & kErrSteps)
        return fail(PARDNN_E_INVAL, "step_ptr must start at 0, never decrease and end at n_moves");
    return PARDNN_OK;
}

int pardnn_evaluate_batch(pardnn_graph *h, int32_t n_place, const int32_t *placements,
                          int32_t n_labels, const int64_t *capacity, int64_t *tl, int64_t *bl,
                          int64_t *makespan, uint8_t *is_critical, int32_t *path,
                          int32_t path_stride, int32_t *path_len, int64_t *label_mem,
                          int64_t *overflow) {
    CHECK_HANDLE(h);
    Graph *g = reinterpret_cast<Graph *>(h);
    if (g->V > 0 && n_place > 0 && placements == nullptr)
        return fail(PARDNN_E_INVAL, "placements must be non-null");
    return evaluate_impl(g, n_place, placements, nullptr, n_labels, capacity, tl, bl, makespan,
                         is_critical, path, path_stride, path_len, label_mem, overflow);
}

int pardnn_evaluate_moves(pardnn_graph *h, const int32_t *base, int32_t n_place,
                          const int64_t *step_ptr, int64_t n_moves, const int32_t *node,
                          const int32_t *label,
                          int32_t n_labels, const int64_t *capacity, int64_t *tl, int64_t *bl,
                          int64_t *makespan, uint8_t *is_critical, int32_t *path,
                          int32_t path_stride, int32_t *path_len, int64_t *label_mem,
                          int64_t *overflow) {
    CHECK_HANDLE(h);
    Graph *g = reinterpret_cast<Graph *>(h);
    if (n_place > 0 && step_ptr == nullptr) return fail(PARDNN_E_INVAL, "step_ptr must be non-null");
    MovesIn mv{base, step_ptr, n_moves, node, label};
    return evaluate_impl(g, n_place, nullptr, &mv, n_labels, capacity, tl, bl, makespan,
                         is_critical, path, path_stride, path_len, label_mem, overflow);
}

int pardnn_set_deferred_errors(pardnn_graph *h, int enable) {
    CHECK_HANDLE(h);
    Graph *g = reinterpret_cast<Graph *>(h);
    DEVICE_SCOPE(g);
    // a fresh start either way: no flags from before the switch
    HIP_TRY(launch_fill_i32(g->err, 1, 0, g->stream));
    g->defer_errors = enable != 0;
    return PARDNN_OK;
}

int pardnn_take_errors(pardnn_graph *h) {
    CHECK_HANDLE(h);
    Graph *g = reinterpret_cast<Graph *>(h);
    DEVICE_SCOPE(g);
    if (!g->defer_errors) {   // every call has reported its own errors already
        HIP_TRY(hipStreamSynchronize(g->stream));
        return PARDNN_OK;
    }
    int32_t flags = 0;
    HIP_TRY(hipMemcpyAsync(&flags, g->err, sizeof(int32_t), hipMemcpyDeviceToHost, g->stream));
    HIP_TRY(hipStreamSynchronize(g->stream));
    HIP_TRY(launch_fill_i32(g->err, 1, 0, g->stream));
    if (flags != 0)
        return fail(PARDNN_E_INVAL, "a call made since the last take found an argument out of "
                                    "range on the device (error flags " +
                                        std::to_string(flags) + ")");
    return PARDNN_OK;
}

int pardnn_set_timing(pardnn_graph *h, int enable) {
    CHECK_HANDLE(h);
    Graph *g = reinterpret_cast<Graph *>(h);
    DEVICE_SCOPE(g);
    if (enable && !g->ev0) {
        HIP_TRY(hipEventCreate(&g->ev0));
        HIP_TRY(hipEventCreate(&g->ev1));
    }
    g->timing = enable != 0;
    g->timed = false;
    return PARDNN_OK;
}

int pardnn_get_timing(pardnn_graph *h, const char **kernel, float *ms) {
    CHECK_HANDLE(h);
    Graph *g = reinterpret_cast<Graph *>(h);
    if (ms == nullptr) return fail(PARDNN_E_INVAL, "ms is null");
    if (!g->timed) return fail(PARDNN_E_INVAL, "no timed launch recorded");
    DEVICE_SCOPE(g);
    HIP_TRY(hipEventSynchronize(g->ev1));
    HIP_TRY(hipEventElapsedTime(ms, g->ev0, g->ev1));
    if (kernel) *kernel = g->timed_kernel;
    return PARDNN_OK;
}

int pardnn_evaluate_batch_fixed(pardnn_graph *h, int32_t n_place, const int32_t *placements,
                                int32_t n_labels, const int64_t *capacity, int64_t *tl,
                                int64_t *bl, int64_t *makespan, uint8_t *is_critical,
                                int32_t *path, int32_t path_stride, int32_t *path_len,
                                int64_t *label_mem, int64_t *overflow) {
    CHECK_HANDLE(h);
    Graph *g = reinterpret_cast<Graph *>(h);
    if (g->V > 0 && n_place > 0 && placements == nullptr)
        return fail(PARDNN_E_INVAL, "placements must be non-null");
    DEVICE_SCOPE(g);
    void *ws = nullptr;
    const int st = fixed_scratch(g->device, &ws);
    if (st != PARDNN_OK) return st;
    return evaluate_impl(g, n_place, placements, nullptr, n_labels, capacity, tl, bl, makespan,
                         is_critical, path, path_stride, path_len, label_mem, overflow, ws,
                         kFixedScratchBytes);
}

int pardnn_tb_levels_batch(pardnn_graph *h, int32_t n_place, const int32_t *placements,
                           int64_t *tl, int64_t *bl, int64_t *makespan) {
    return pardnn_evaluate_batch(h, n_place, placements, 0, nullptr, tl, bl, makespan, nullptr,
                                 nullptr, 0, nullptr, nullptr, nullptr);
}

}  // extern "C"
