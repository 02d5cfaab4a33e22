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
// trip per level. A wide frontier is expanded by the whole workgroup, edge-
// parallel: a workgroup scan of the frontier's out-degrees maps every thread
// to one out-edge, so a single high-fan-out node does not serialise on one
// lane. An in-degree counter that reaches zero appends its node to the next
// frontier (an LDS counter) and loads its out-edge range into LDS right away.
// A frontier of at most 8 nodes -- the long one-wide chains of deep graphs --
// is walked by one wave alone, level after level, without workgroup
// barriers: every node carries a 32-byte record with its first six
// successors, so such a level is two memory round trips (the in-degree
// decrements of the frontier's successors, then the records of the nodes
// they release); the successors past the sixth are spread over the wave in
// chunks of 64. The wave hands the frontier back to the workgroup when it
// widens. The workgroup's own levels count their releases in two alternating
// LDS counters, so a level needs three workgroup barriers. `level_ptr` falls
// out of the frontier sizes; `order` -- ids sorted by (level, id) -- comes
// from one stable radix sort of the levels afterwards.

#include <algorithm>

#include "device_utils.h"
#include "internal.h"

namespace pardnn {

namespace {

constexpr int KT = 1024;     // threads of the Kahn workgroup
constexpr int kCap = 1024;   // frontier entries whose records live in LDS

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

constexpr int kInl = 6;       // successors held in a node's record
constexpr int kNarrow = 8;    // frontiers of at most this many nodes go to one wave

// A node's out-edge range and its first kInl successors (original ids).
struct alignas(16) KahnRec {
    int32_t e0, deg;
    int32_t s[kInl];
};
static_assert(sizeof(KahnRec) == 32, "two 16-byte loads per node");

__global__ void k_kahn_recs(int32_t V, const int32_t *o_off, const int32_t *o_nbr,
                            KahnRec *rec) {
    for (int32_t v = blockIdx.x * blockDim.x + threadIdx.x; v < V; v += gridDim.x * blockDim.x) {
        KahnRec r;
        r.e0 = o_off[v];
        r.deg = o_off[v + 1] - r.e0;
#pragma unroll
        for (int k = 0; k < kInl; k++) r.s[k] = k < r.deg ? o_nbr[r.e0 + k] : -1;
        rec[v] = r;
    }
}

// Wave 0 alone walks levels while the frontier holds at most 64 nodes.
// Entry: the frontier is queue[head, tail) (level L - 1); s_nf holds it when
// `in_lds`. Exit: (head, tail, L) in st[0..2] for the workgroup.
__device__ void kahn_narrow(const int32_t *o_nbr, const KahnRec *rec, int32_t *indeg,
                            int32_t *queue, int32_t *level_ptr, int32_t *level, int32_t head,
                            int32_t tail, int32_t L, int32_t *s_nf, int32_t *s_xoff,
                            int32_t *s_xe0, int32_t *st) {
    const int lane = lane_id();
    const unsigned long long below = (1ull << lane) - 1ull;
    int32_t nf = tail - head;
    int32_t u = lane < nf ? queue[head + lane] : -1;
    while (nf > 0 && nf <= kNarrow) {
        // the frontier's records: offset, degree, first successors
        KahnRec r;
        if (u >= 0) {
            r = rec[u];
        } else {
            r.e0 = 0;
            r.deg = 0;
        }
        int32_t n_next = 0;
        auto release = [&](bool rel, int32_t t) {
            const unsigned long long m = __ballot(rel);
            if (rel) {
                const int32_t pos = n_next + __popcll(m & below);
                queue[tail + pos] = t;
                level[t] = L;
                if (pos < kWave) s_nf[pos] = t;
            }
            n_next += __popcll(m);
        };
        // successors past the inline ones, flattened over the wave: lane l
        // holds extra edges [xoff, xoff + xdeg) of the list; an edge's owner
        // is found by binary search over the lanes' offsets in LDS
        const int32_t xdeg = r.deg > kInl ? r.deg - kInl : 0;
        int32_t xtot = 0;
        if (__ballot(xdeg > 0) != 0ull) {
            const int32_t xincl = wave_incl_scan_i32(xdeg);
            xtot = __builtin_amdgcn_readlane(xincl, kWave - 1);
            s_xoff[lane] = xincl - xdeg;
            s_xe0[lane] = r.e0 + kInl;
        }
        auto extra = [&](int32_t j) -> int32_t {   // the j-th extra successor, or -1
            if (j >= xtot) return -1;
            int lo = 0, hi = kWave;   // s_xoff[lo] <= j < s_xoff[hi] (hi = 64: end)
            while (hi - lo > 1) {
                const int mid = (lo + hi) >> 1;
                if (s_xoff[mid] <= j)
                    lo = mid;
                else
                    hi = mid;
            }
            return o_nbr[s_xe0[lo] + (j - s_xoff[lo])];
        };
        // the first 64 extra successors load while the inline ones decrement
        int32_t t2 = xtot > 0 ? extra(lane) : -1;
        int32_t t[kInl], old[kInl];
#pragma unroll
        for (int k = 0; k < kInl; k++) t[k] = k < r.deg ? r.s[k] : -1;
#pragma unroll
        for (int k = 0; k < kInl; k++) old[k] = t[k] >= 0 ? atomicSub(&indeg[t[k]], 1) : 0;
#pragma unroll
        for (int k = 0; k < kInl; k++) release(t[k] >= 0 && old[k] == 1, t[k]);
        for (int32_t c0 = 0; c0 < xtot; c0 += kWave) {
            if (c0 > 0) t2 = extra(c0 + lane);
            const int32_t o2 = t2 >= 0 ? atomicSub(&indeg[t2], 1) : 0;
            release(t2 >= 0 && o2 == 1, t2);
        }
        head = tail;
        tail += n_next;
        nf = n_next;
        if (n_next > 0) {
            L++;
            if (lane == 0) level_ptr[L] = tail;
        }
        if (nf > kNarrow) break;
        u = lane < nf ? s_nf[lane] : -1;
    }
    if (lane == 0) {
        st[0] = head;
        st[1] = tail;
        st[2] = L;
    }
}

__global__ __launch_bounds__(KT) void k_kahn(int32_t V, const int32_t *o_off,
                                             const int32_t *o_nbr, const KahnRec *rec,
                                             int32_t *indeg, int32_t *queue, int32_t *level_ptr,
                                             int32_t *level, int32_t *result) {
    // records (out-edge range, first successors) of the first kCap nodes of
    // the current and the next frontier, loaded when a node is released
    __shared__ KahnRec s_rec[2][kCap];
    __shared__ int32_t s_off[KT];
    __shared__ int32_t s_base[KT];
    __shared__ int wsum[KT / kWave + 1];
    __shared__ int32_t s_cnt[2];
    __shared__ int32_t s_nf[kWave], s_xoff[kWave], s_xe0[kWave];
    __shared__ int32_t s_st[3];
    const int tid = threadIdx.x;
    bool staged = true;   // s_e0 / s_deg hold the current frontier's ranges

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
            if (n0 + pos < kCap) s_rec[0][n0 + pos] = rec[v];
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
    if (tid == 0) s_cnt[0] = s_cnt[1] = 0;
    __syncthreads();
    while (tail > head) {
        if (tail - head <= kNarrow) {
            if (wave_id() == 0)
                kahn_narrow(o_nbr, rec, indeg, queue, level_ptr, level, head, tail, L, s_nf,
                            s_xoff, s_xe0, s_st);
            __builtin_amdgcn_s_waitcnt(0);
            __threadfence_block();
            __syncthreads();
            head = s_st[0];
            tail = s_st[1];
            L = s_st[2];
            staged = false;   // the widened frontier's ranges are not in LDS
            __syncthreads();
            continue;
        }
        for (int32_t cb = head; cb < tail; cb += KT) {
            const int nf = min(KT, tail - cb);
            const int32_t idx = cb - head + tid;   // position in the frontier
            // frontier nodes whose records are staged in LDS read their first
            // successors there; the others read the CSR
            const bool in_lds = staged && cb - head + KT <= kCap;
            int deg = 0;
            int32_t e0 = 0;
            if (tid < nf) {
                if (in_lds) {
                    e0 = s_rec[cur][idx].e0;
                    deg = s_rec[cur][idx].deg;
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
                const int t = owner_of(s_off, nf, j);
                const int32_t k = j - s_off[t];
                const int32_t s = in_lds && k < kInl ? s_rec[cur][cb - head + t].s[k]
                                                     : o_nbr[s_base[t] + k];
                const int32_t old = atomicSub(&indeg[s], 1);
                if (old == 1) {
                    const int32_t p = atomicAdd(&s_cnt[cur], 1);
                    queue[tail + p] = s;
                    level[s] = L;
                    if (p < kCap) s_rec[cur ^ 1][p] = rec[s];
                }
            }
            __syncthreads();
        }
        // every thread has passed the barrier that closed the edge loop, and
        // read the other counter before this level's first barrier: it can
        // be cleared for the next level without another barrier
        const int32_t n_next = s_cnt[cur];
        if (tid == 0) s_cnt[cur ^ 1] = 0;
        head = tail;
        tail += n_next;
        cur ^= 1;
        staged = true;
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
size_t kahn_rec_bytes(int32_t V) { return (size_t)std::max(V, 1) * sizeof(KahnRec); }

hipError_t launch_kahn(const Graph &g, int32_t *indeg_work, int32_t *queue, int32_t *result,
                       void *rec_scratch) {
    KahnRec *rec = reinterpret_cast<KahnRec *>(rec_scratch);
    if (g.V > 0) {
        const unsigned grid = (unsigned)std::min<int64_t>((g.V + 255) / 256, 65536);
        k_kahn_recs<<<grid, 256, 0, g.stream>>>(g.V, g.o_off, g.o_nbr, rec);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    k_kahn<<<1, KT, 0, g.stream>>>(g.V, g.o_off, g.o_nbr, rec, indeg_work, queue, g.level_ptr,
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
