// levelize.hip -- topological levels by Kahn's algorithm in one persistent
// workgroup.
//
// The paper obtains weighted levels by a topological-order pass costing
// O(|V| + |E|) (Sec. 3.1.1, complexity of Alg. 1) and indexes per-level
// work by level (Sec. 3.1.2, Fenwick trees over levels). Here level(v) is the
// Kahn frontier index: 0 without predecessors, else 1 + max over predecessors.
//
// Design for gfx950: the frontier loop is a chain of dependent steps (one per
// level, ~100k of them for deep graphs), so it runs inside ONE workgroup with
// only workgroup barriers between levels -- no kernel launch and no host round
// trip per level. Each step is edge-parallel: a workgroup scan of the
// frontier's out-degrees maps every thread to one out-edge, so a single
// high-fan-out node does not serialise on one lane. An in-degree counter that
// reaches zero appends its node to the next frontier (an LDS counter) and
// loads its out-edge range into LDS right away, so the next level starts
// without a dependent global load. `level_ptr` falls out of the frontier
// sizes; `order` -- ids sorted by (level, id) -- comes from one stable radix
// sort of the levels afterwards instead of a sort per level.

#include "device_utils.h"
#include "internal.h"

namespace pardnn {

namespace {

constexpr int KT = 1024;     // threads of the Kahn workgroup
constexpr int kCap = 2048;   // frontier entries whose out-edge ranges live in LDS

// Largest t in [0, n) with off[t] <= j (off non-decreasing, off[0] == 0).
__device__ __forceinline__ int owner_of(const int32_t *off, int n, int32_t j) {
    int lo = 0, hi = n;  // invariant: off[lo] <= j, answer in [lo, hi)
    while (hi - lo > 1) {
        int mid = (lo + hi) >> 1;
        if (off[mid] <= j)
            lo = mid;
        else
            hi = mid;
    }
    return lo;
}

__global__ __launch_bounds__(KT) void k_kahn(int32_t V, const int32_t *o_off,
                                             const int32_t *o_nbr, int32_t *indeg,
                                             int32_t *queue, int32_t *level_ptr,
                                             int32_t *level, int32_t *result) {
    // out-edge range (start, count) of the first kCap nodes of the current and
    // the next frontier, loaded when a node is released
    __shared__ int32_t s_e0[2][kCap], s_deg[2][kCap];
    __shared__ int32_t s_off[KT];
    __shared__ int32_t s_base[KT];
    __shared__ int wsum[KT / kWave + 1];
    __shared__ int32_t s_cnt;
    const int tid = threadIdx.x;

    // Level 0: nodes without predecessors, compacted in id order.
    int32_t n0 = 0;
    for (int32_t b = 0; b < V; b += KT) {
        int32_t v = b + tid;
        int f = (v < V && indeg[v] == 0) ? 1 : 0;
        int total;
        int pos = block_excl_scan_i32(f, wsum, &total);
        if (f) {
            queue[n0 + pos] = v;
            level[v] = 0;
            if (n0 + pos < kCap) {
                const int32_t a = o_off[v];
                s_e0[0][n0 + pos] = a;
                s_deg[0][n0 + pos] = o_off[v + 1] - a;
            }
        }
        n0 += total;
        __syncthreads();
    }
    int32_t L = 0;
    if (tid == 0) level_ptr[0] = 0;
    if (n0 > 0) {
        L = 1;
        if (tid == 0) level_ptr[1] = n0;
    }
    int32_t head = 0, tail = n0;
    int cur = 0;
    while (tail > head) {
        if (tid == 0) s_cnt = 0;
        __syncthreads();
        for (int32_t cb = head; cb < tail; cb += KT) {
            const int nf = min(KT, tail - cb);
            const int32_t idx = cb - head + tid;   // position in the frontier
            int deg = 0;
            int32_t e0 = 0;
            if (tid < nf) {
                if (idx < kCap) {
                    e0 = s_e0[cur][idx];
                    deg = s_deg[cur][idx];
                } else {
                    const int32_t u = queue[cb + tid];
                    e0 = o_off[u];
                    deg = o_off[u + 1] - e0;
                }
            }
            int total;
            int ex = block_excl_scan_i32(deg, wsum, &total);
            s_off[tid] = ex;
            s_base[tid] = e0;
            __syncthreads();
            for (int32_t j = tid; j < total; j += KT) {
                int t = owner_of(s_off, nf, j);
                int32_t s = o_nbr[s_base[t] + (j - s_off[t])];
                int32_t old = atomicSub(&indeg[s], 1);
                if (old == 1) {
                    int32_t p = atomicAdd(&s_cnt, 1);
                    queue[tail + p] = s;
                    level[s] = L;
                    if (p < kCap) {
                        const int32_t a = o_off[s];
                        s_e0[cur ^ 1][p] = a;
                        s_deg[cur ^ 1][p] = o_off[s + 1] - a;
                    }
                }
            }
            __syncthreads();
        }
        const int32_t n_next = s_cnt;
        __syncthreads();
        head = tail;
        tail += n_next;
        cur ^= 1;
        if (n_next > 0) {
            L++;
            if (tid == 0) level_ptr[L] = tail;
        }
    }
    if (tid == 0) {
        result[0] = L;
        result[1] = tail;
    }
}

}  // namespace

// result[0] = number of levels, result[1] = nodes released (< V: cycle);
// `queue` (int32[V]) receives the nodes in release order.
hipError_t launch_kahn(const Graph &g, int32_t *indeg_work, int32_t *queue, int32_t *result) {
    k_kahn<<<1, KT, 0, g.stream>>>(g.V, g.o_off, g.o_nbr, indeg_work, queue, g.level_ptr,
                                   g.level, result);
    return hipGetLastError();
}

size_t level_order_scratch_bytes(int32_t V) {
    return ((size_t)V * 8 + 255) / 256 * 256 + sort_pairs_scratch_bytes(V, 4);
}

// order = node ids sorted by (level, id): a stable radix sort of the levels
// (low `bits` bits) over the ids given in ascending order.
hipError_t launch_level_order(const Graph &g, int32_t bits, void *scratch) {
    const int32_t V = g.V;
    if (V == 0) return hipSuccess;
    const size_t head = ((size_t)V * 8 + 255) / 256 * 256;
    int32_t *ids = reinterpret_cast<int32_t *>(scratch);
    uint32_t *keys_out = reinterpret_cast<uint32_t *>(ids + V);
    void *temp = reinterpret_cast<char *>(scratch) + head;
    hipError_t e = launch_iota_i32(ids, V, g.stream);
    if (e != hipSuccess) return e;
    return sort_pairs_u32(reinterpret_cast<const uint32_t *>(g.level), keys_out, ids, g.order, V,
                          0, bits, temp, g.stream);
}

}  // namespace pardnn
