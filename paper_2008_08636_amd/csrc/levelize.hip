// levelize.hip -- topological levels by Kahn's algorithm in one persistent
// workgroup.
//
// The paper computes weighted levels with "a variant of topological sorting"
// in O(|V| + |E|) (Sec. 3.1.1, complexity of Alg. 1) and indexes per-level
// work by level (Sec. 3.1.2, Fenwick trees over levels). Here level(v) is the
// Kahn frontier index: 0 without predecessors, else 1 + max over predecessors.
//
// Design for gfx950: the frontier loop is a chain of dependent steps (one per
// level, ~100k of them for deep graphs), so it runs inside ONE workgroup with
// only workgroup barriers between levels -- no kernel launch and no host round
// trip per level. Each step is edge-parallel: a workgroup scan of the
// frontier's out-degrees maps every thread to one out-edge, so a single
// high-fan-out node does not serialise on one lane. An in-degree counter that
// reaches zero appends its node to the next frontier (an LDS counter), which
// is then sorted by id in LDS (bitonic), so `order` comes out sorted by
// (level, id) and `level_ptr` falls out of the frontier sizes.
#include "device_utils.h"
#include "internal.h"

namespace pardnn {

namespace {

constexpr int KT = 1024;             // threads of the Kahn workgroup
constexpr int kSortCap = 8192;       // largest frontier sorted in LDS

__device__ __forceinline__ void bitonic_step(int32_t *key, int n, int size, int stride) {
    for (int i = threadIdx.x; i < n / 2; i += KT) {
        int lo = (i / stride) * stride * 2 + (i % stride);
        int hi = lo + stride;
        bool asc = (lo & size) == 0;
        int32_t x = key[lo], y = key[hi];
        if ((x > y) == asc) {
            key[lo] = y;
            key[hi] = x;
        }
    }
}

// Sort seg[0..n) ascending. n <= kSortCap: in LDS; otherwise in `scratch`
// (global, at least next_pow2(n) ints), with the same network.
__device__ void sort_segment(int32_t *seg, int n, int32_t *lds, int32_t *scratch) {
    int m = 1;
    while (m < n) m <<= 1;
    int32_t *key = m <= kSortCap ? lds : scratch;
    for (int i = threadIdx.x; i < m; i += KT) key[i] = i < n ? seg[i] : INT32_MAX;
    __syncthreads();
    for (int size = 2; size <= m; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            bitonic_step(key, m, size, stride);
            __syncthreads();
        }
    }
    for (int i = threadIdx.x; i < n; i += KT) seg[i] = key[i];
    __syncthreads();
}

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
                                             int32_t *order, int32_t *level_ptr,
                                             int32_t *level, int32_t *sort_scratch,
                                             int32_t *result) {
    __shared__ int32_t s_key[kSortCap];
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
            order[n0 + pos] = v;
            level[v] = 0;
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
    while (tail > head) {
        if (tid == 0) s_cnt = 0;
        __syncthreads();
        for (int32_t cb = head; cb < tail; cb += KT) {
            const int nf = min(KT, tail - cb);
            int32_t i = cb + tid;
            int deg = 0;
            int32_t e0 = 0;
            if (tid < nf) {
                int32_t u = order[i];
                e0 = o_off[u];
                deg = o_off[u + 1] - e0;
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
                    order[tail + p] = s;
                    level[s] = L;
                }
            }
            __syncthreads();
        }
        const int32_t n_next = s_cnt;
        __syncthreads();
        if (n_next > 1) sort_segment(order + tail, n_next, s_key, sort_scratch);
        head = tail;
        tail += n_next;
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

// result[0] = number of levels, result[1] = nodes released (< V: cycle).
hipError_t launch_kahn(const Graph &g, int32_t *indeg_work, int32_t *sort_scratch,
                       int32_t *result) {
    k_kahn<<<1, KT, 0, g.stream>>>(g.V, g.o_off, g.o_nbr, indeg_work, g.order, g.level_ptr,
                                   g.level, sort_scratch, result);
    return hipGetLastError();
}

}  // namespace pardnn
