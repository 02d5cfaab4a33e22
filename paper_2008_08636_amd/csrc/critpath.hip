// critpath.hip -- critical nodes and the canonical critical path for one
// placement (paper Table 2, CP; Alg. 1 find_heaviest_path walking by weighted
// level on fresh values).
//
//   is_critical(v) = (tl(v) + bl(v) == M)
//   next(u)        = smallest-id successor s with tl(u)+comp(u)+c(u,s)+bl(s) == M
//   path           = smallest-id critical node without predecessors, then next()
//                    until a node without a tight successor.
//
// Design for gfx950: next() of every node is one data-parallel pass over the
// out-edges (level-major CSR). When the critical nodes form one chain (one
// critical path) the path is their list in level-major order, found by a
// scan and checked link by link in parallel. Otherwise the walk is a pointer
// chase, and its
// links only point to strictly later levels, i.e. to larger level-major ids.
// One workgroup therefore stages a window of next() in LDS with a coalesced
// load, chases inside the window at LDS latency, and reloads the window only
// when the chase leaves it -- the window only ever moves forward.
#include "device_utils.h"
#include "internal.h"

namespace pardnn {

namespace {

constexpr int kBlock = 256;
constexpr int kChaseThreads = 1024;
constexpr int kWindow = 8192;

inline unsigned grid_for(int64_t n, int block, int cap = 65536) {
    int64_t g = (n + block - 1) / block;
    if (g < 1) g = 1;
    if (g > cap) g = cap;
    return (unsigned)g;
}

// Additions wrap instead of overflowing for inputs not produced by the sweep;
// for consistent inputs every sum stays below the ingest bound.
__device__ __forceinline__ int64_t wadd(int64_t a, int64_t b) {
    return (int64_t)((uint64_t)a + (uint64_t)b);
}

// Critical flags per node; the next-hop slot starts empty.
__global__ void k_crit_flags(int32_t V, const int32_t *order, const int64_t *tl,
                             const int64_t *bl, const int64_t *makespan, uint8_t *is_critical,
                             int32_t *next_lm, uint8_t *crit_lm) {
    const int64_t M = *makespan;
    for (int32_t v = blockIdx.x * blockDim.x + threadIdx.x; v < V; v += gridDim.x * blockDim.x) {
        const int32_t ov = order[v];
        const uint8_t crit = wadd(tl[ov], bl[ov]) == M;
        is_critical[ov] = crit;
        crit_lm[v] = crit;
        next_lm[v] = INT32_MAX;
    }
}

// One thread per out-edge (level-major): a tight edge offers its successor's
// original id to its source; the smallest wins. Every node gets its next hop,
// critical or not: the walk's definition steps along tight edges from any node
// it reaches, which matters for tl / bl that no sweep produced. Edge-parallel,
// so a node with thousands of successors costs no more than as many edges.
__global__ void k_crit_tight(int64_t E, const int32_t *order, const int32_t *out_src,
                             const int32_t *out_dst_orig, const int64_t *out_cost,
                             const int64_t *comp_lm, const int32_t *placement, const int64_t *tl,
                             const int64_t *bl, const int64_t *makespan, int32_t *next_lm) {
    const int64_t M = *makespan;
    for (int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; j < E;
         j += (int64_t)gridDim.x * blockDim.x) {
        const int32_t v = out_src[j];
        const int32_t ov = order[v], so = out_dst_orig[j];
        const int64_t c = placement[ov] != placement[so] ? out_cost[j] : 0;
        if (wadd(wadd(wadd(tl[ov], comp_lm[v]), c), bl[so]) == M) atomicMin(&next_lm[v], so);
    }
}

// original id of the chosen successor -> its level-major index (-1: none)
__global__ void k_crit_link(int32_t V, const int32_t *rank, int32_t *next_lm) {
    for (int32_t v = blockIdx.x * blockDim.x + threadIdx.x; v < V; v += gridDim.x * blockDim.x) {
        const int32_t o = next_lm[v];
        next_lm[v] = o == INT32_MAX ? -1 : rank[o];
    }
}

// The walk starts at the smallest-id critical node without predecessors, or,
// when start_orig is given, at that node (INT32_MAX: no path).
__global__ __launch_bounds__(kChaseThreads) void k_chase(int32_t V, int32_t n0,
                                                         const int32_t *order,
                                                         const int32_t *rank,
                                                         const int32_t *start_orig,
                                                         const int32_t *next_lm,
                                                         const uint8_t *crit_lm, int32_t *path,
                                                         int32_t *path_len, const int32_t *done) {
    if (done != nullptr && *done) return;   // the list pass already wrote the path
    __shared__ int32_t win[kWindow];
    __shared__ int s_start, s_cur, s_len;
    const int tid = threadIdx.x;
    if (tid == 0) {
        s_start = INT32_MAX;
        s_len = 0;
    }
    __syncthreads();
    // level 0 is sorted by original id: the smallest critical lm index there
    // is the smallest-id critical node without predecessors
    if (start_orig == nullptr) {
        for (int32_t v = tid; v < n0; v += kChaseThreads)
            if (crit_lm[v]) lds_min_i32(&s_start, v);
    } else if (tid == 0 && *start_orig != INT32_MAX) {
        s_start = rank[*start_orig];
    }
    __syncthreads();
    if (tid == 0) s_cur = s_start == INT32_MAX ? -1 : s_start;
    __syncthreads();
    while (true) {
        const int32_t base = s_cur;
        if (base < 0) break;
        for (int i = tid; i < kWindow; i += kChaseThreads)
            win[i] = base + i < V ? next_lm[base + i] : -1;
        __syncthreads();
        if (tid == 0) {
            int32_t c = base, len = s_len;
            while (c >= base && c < base + kWindow) {
                path[len++] = order[c];
                int32_t n = win[c - base];
                // links go to strictly later levels; anything else ends the walk
                c = n > c ? n : -1;
            }
            s_cur = c;
            s_len = len;
        }
        __syncthreads();
    }
    if (tid == 0) *path_len = s_len;
}

// The list pass: when the critical nodes, in level-major order, form one
// chain -- each links to the next, the last to nothing, and the first is the
// walk's start -- that list is the path (the usual case: one critical path).
// Then the path is written in parallel and the walk returns at once.
__global__ void k_path_flags(int32_t V, const uint8_t *crit_lm, int32_t *f) {
    for (int32_t v = blockIdx.x * blockDim.x + threadIdx.x; v < V; v += gridDim.x * blockDim.x)
        f[v] = crit_lm[v] ? 1 : 0;
}

__global__ void k_path_list(int32_t V, const uint8_t *crit_lm, const int32_t *pos,
                            int32_t *list) {
    for (int32_t v = blockIdx.x * blockDim.x + threadIdx.x; v < V; v += gridDim.x * blockDim.x)
        if (crit_lm[v]) list[pos[v]] = v;
}

// ok = 1 beforehand; n = pos[V] critical nodes
__global__ void k_path_check(int32_t V, int32_t n0, const int32_t *pos, const int32_t *list,
                             const int32_t *next_lm, const int32_t *rank,
                             const int32_t *start_orig, int32_t *ok) {
    const int32_t n = pos[V];
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
        const int32_t want = i + 1 < n ? list[i + 1] : -1;
        if (next_lm[list[i]] != want) *ok = 0;
    }
    if (blockIdx.x == 0 && threadIdx.x == 0 && n > 0) {
        bool start_ok;
        if (start_orig == nullptr) {
            start_ok = list[0] < n0;   // level 0 is sorted by id
        } else {
            const int32_t s = *start_orig;
            start_ok = s != INT32_MAX && rank[s] == list[0];
        }
        if (!start_ok) *ok = 0;
    }
}

__global__ void k_path_write(int32_t V, const int32_t *pos, const int32_t *list,
                             const int32_t *order, const int32_t *ok, int32_t *path,
                             int32_t *path_len) {
    if (!*ok) return;
    const int32_t n = pos[V];
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x)
        path[i] = order[list[i]];
    if (blockIdx.x == 0 && threadIdx.x == 0) *path_len = n;
}

}  // namespace

hipError_t launch_crit_next(const Graph &g, const int32_t *placement, const int64_t *comp_lm,
                            const int64_t *tl, const int64_t *bl, const int64_t *makespan,
                            uint8_t *is_critical) {
    if (g.V == 0) return hipSuccess;
    k_crit_flags<<<grid_for(g.V, kBlock), kBlock, 0, g.stream>>>(
        g.V, g.order, tl, bl, makespan, is_critical, g.next_lm, g.crit_lm);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (g.E > 0) {
        k_crit_tight<<<grid_for(g.E, kBlock), kBlock, 0, g.stream>>>(
            g.E, g.order, g.out_src, g.out_dst_orig, g.out_cost, comp_lm, placement, tl, bl,
            makespan, g.next_lm);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    k_crit_link<<<grid_for(g.V, kBlock), kBlock, 0, g.stream>>>(g.V, g.rank, g.next_lm);
    return hipGetLastError();
}

hipError_t launch_chase_from(const Graph &g, const int32_t *start_orig, int32_t *path,
                             int32_t *path_len) {
    const int32_t n0 = g.L > 0 ? g.h_level_ptr[1] : 0;
    const int32_t V = g.V;
    int32_t *ok = g.cp_ok;
    hipError_t e = launch_fill_i32(ok, 1, 1, g.stream);
    if (e != hipSuccess) return e;
    if (V > 0) {
        k_path_flags<<<grid_for(V, kBlock), kBlock, 0, g.stream>>>(V, g.crit_lm, g.cp_flag);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if ((e = launch_exclusive_scan(g.cp_flag, g.cp_pos, V, g.cp_ws, g.stream)) != hipSuccess)
            return e;
        k_path_list<<<grid_for(V, kBlock), kBlock, 0, g.stream>>>(V, g.crit_lm, g.cp_pos,
                                                                 g.cp_list);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        k_path_check<<<grid_for(V, kBlock), kBlock, 0, g.stream>>>(
            V, n0, g.cp_pos, g.cp_list, g.next_lm, g.rank, start_orig, ok);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        k_path_write<<<grid_for(V, kBlock), kBlock, 0, g.stream>>>(V, g.cp_pos, g.cp_list,
                                                                  g.order, ok, path, path_len);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    k_chase<<<1, kChaseThreads, 0, g.stream>>>(V, n0, g.order, g.rank, start_orig, g.next_lm,
                                               g.crit_lm, path, path_len, V > 0 ? ok : nullptr);
    return hipGetLastError();
}

hipError_t launch_critical_path(const Graph &g, const int32_t *placement, const int64_t *tl,
                                const int64_t *bl, const int64_t *makespan,
                                uint8_t *is_critical, int32_t *path, int32_t *path_len) {
    hipError_t e = launch_crit_next(g, placement, g.comp_lm, tl, bl, makespan, is_critical);
    if (e != hipSuccess) return e;
    return launch_chase_from(g, nullptr, path, path_len);
}

}  // namespace pardnn
