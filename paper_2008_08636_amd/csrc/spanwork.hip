// spanwork.hip -- the terms of level-aware load balancing (paper Eq. 2, Sec.
// 3.1.2) for a batch of secondary clusters against the current partitions.
//
// For a cluster sc with topologically first node f and last node l, span(sc)
// runs from the latest finish time tl(p) + comp(p) over the parents p of f
// (0 without parents) to the earliest start time tl(c) over the children c of
// l (the makespan max tl + comp without children) -- the span of Table 2.
// Per cluster and partition k:
//   work[sc][k] = sum of comp(n) over nodes n on k with lo <= tl(n) <= hi
//   comm[sc][k] = sum of edge costs between sc and nodes on k (edges inside
//                 one cluster excluded)
//   Eq. 2 cost  = work[sc][k] + (sum over k' of comm[sc][k']) - comm[sc][k]
// and the choice is the partition of least cost, ties to the largest comm,
// then to the smallest k.
//
// Design for gfx950: the paper keeps per-level weights in Fenwick trees so the
// sequential mapping loop can query one span at a time. Here all queries of a
// batch run at once, so the table is static: the mapped nodes sorted by
// (partition, tl) with a prefix sum of their weights, after which one span
// query is two binary searches in its partition's segment. The nodes in
// (tl, id) order are kept on the graph handle with a copy of the tl they came
// from: the mapping loop calls again with the same tl and new partitions, so
// a call compares tl with the copy on the device and re-sorts by tl (a 64-bit
// radix sort, its launches gated by the comparison) only when it changed;
// every call then splits that order by partition with a one-pass stable
// radix sort. The communication table and the span ends are passes of 64-bit
// atomics over the edge list (edge-parallel, so hub nodes with thousands of
// edges cost no serial loop); cluster ends are 64-bit atomic min / max of
// (level, id) keys.
#include <climits>

#include <algorithm>

#include "device_utils.h"
#include "internal.h"

namespace pardnn {

namespace {

constexpr int kBlock = 256;

inline unsigned grid_for(int64_t n, int block, int cap = 65536) {
    int64_t g = (n + block - 1) / block;
    if (g < 1) g = 1;
    if (g > cap) g = cap;
    return (unsigned)g;
}

inline size_t align256(size_t b) { return (b + 255) / 256 * 256; }

// Scratch layout for V nodes, C clusters, K partitions.
struct SwLayout {
    size_t ids0, ids1, tl_key, tl_key_out, lab_key, lab_sorted, s_tl, w, pre, seg, first, last,
        m, temp, total;
    SwLayout(int32_t V, int32_t C, int32_t K) {
        size_t o = 0;
        auto take = [&](size_t bytes) {
            size_t at = o;
            o += align256(bytes);
            return at;
        };
        ids0 = take((size_t)V * 4);
        ids1 = take((size_t)V * 4);
        tl_key = take((size_t)V * 8);
        tl_key_out = take((size_t)V * 8);
        lab_key = take((size_t)V * 4);
        lab_sorted = take((size_t)V * 4);
        s_tl = take((size_t)V * 8);
        w = take((size_t)V * 8);
        pre = take((size_t)(V + 1) * 8);
        seg = take((size_t)(K + 1) * 4);
        first = take((size_t)C * 8);
        last = take((size_t)C * 8);
        m = take(8);
        size_t t = sort_pairs_scratch_bytes(V, 8);
        t = std::max(t, inclusive_scan_i64_scratch_bytes(V));
        temp = take(t);
        total = o;
    }
};

template <class T>
T *at(void *base, size_t off) {
    return reinterpret_cast<T *>(reinterpret_cast<char *>(base) + off);
}

// Per node: validate ids, cluster ends as (level << 32 | id) keys, the makespan
// max(tl + comp).
__global__ void k_sw_nodes(int32_t V, int32_t K, int32_t C, const int32_t *label,
                           const int32_t *cluster, const int32_t *level, const int64_t *tl,
                           const int64_t *comp, long long *first, long long *last, long long *m,
                           int32_t *err) {
    long long best = LLONG_MIN;
    for (int32_t v = blockIdx.x * blockDim.x + threadIdx.x; v < V; v += gridDim.x * blockDim.x) {
        const int32_t c = cluster[v], k = label[v];
        if (c < -1 || c >= C) atomicOr(err, 1);
        if (k < -1 || k >= K) atomicOr(err, 2);
        if (c >= 0 && c < C) {
            const long long key = ((long long)level[v] << 32) | (long long)v;
            atomicMin(&first[c], key);
            atomicMax(&last[c], key);
        }
        const long long f = tl[v] + comp[v];
        best = f > best ? f : best;
    }
    best = wave_max_i64(best);
    if (lane_id() == 0 && best != LLONG_MIN) atomicMax(m, best);
}

// changed = 1 when tl differs from the copy the cached order was built from
__global__ void k_sw_tl_cmp(int32_t V, const int64_t *tl, const int64_t *copy, int32_t *changed) {
    bool diff = false;
    for (int32_t v = blockIdx.x * blockDim.x + threadIdx.x; v < V; v += gridDim.x * blockDim.x)
        diff = diff || tl[v] != copy[v];
    if (__ballot(diff) != 0ull && lane_id() == 0) *changed = 1;
}

// (when tl changed) sort keys with the order of signed tl, identity values,
// and the new copy of tl
__global__ void k_sw_tl_keys(int32_t V, const int64_t *tl, const int32_t *changed, uint64_t *key,
                             int32_t *ids, int64_t *copy) {
    if (*changed == 0) return;
    for (int32_t v = blockIdx.x * blockDim.x + threadIdx.x; v < V; v += gridDim.x * blockDim.x) {
        const int64_t t = tl[v];
        key[v] = (uint64_t)t ^ (1ull << 63);
        ids[v] = v;
        copy[v] = t;
    }
}

// partition of the i-th node in tl order; unmapped (or invalid) nodes sort last
__global__ void k_sw_lab_keys(int32_t V, int32_t K, const int32_t *label, const int32_t *ids,
                              uint32_t *key) {
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < V; i += gridDim.x * blockDim.x) {
        const int32_t k = label[ids[i]];
        key[i] = (k >= 0 && k < K) ? (uint32_t)k : (uint32_t)K;
    }
}

// nodes in (partition, tl) order: their tl and their weights
__global__ void k_sw_gather(int32_t V, const int32_t *ids, const int64_t *tl,
                            const int64_t *comp, int64_t *s_tl, int64_t *w) {
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < V; i += gridDim.x * blockDim.x) {
        const int32_t v = ids[i];
        s_tl[i] = tl[v];
        w[i] = comp[v];
    }
}

// seg[k] = first position with partition >= k, k = 0..K
__global__ void k_sw_seg(int32_t V, int32_t K, const uint32_t *lab_sorted, int32_t *seg) {
    const int32_t k = blockIdx.x * blockDim.x + threadIdx.x;
    if (k > K) return;
    int32_t lo = 0, hi = V;
    while (lo < hi) {
        const int32_t mid = (lo + hi) >> 1;
        if (lab_sorted[mid] < (uint32_t)k)
            lo = mid + 1;
        else
            hi = mid;
    }
    seg[k] = lo;
}

// span(sc): latest parent finish of the first node (0 without parents),
// earliest child start of the last node (the makespan without children).
// Edge-parallel, so a first or last node with thousands of neighbours costs no
// more than as many edges: init, one pass over the edges, then the defaults.
__global__ void k_sw_bounds_init(int32_t C, const long long *first, long long *lo,
                                 long long *hi) {
    for (int32_t c = blockIdx.x * blockDim.x + threadIdx.x; c < C; c += gridDim.x * blockDim.x) {
        const bool empty = first[c] == LLONG_MAX;
        lo[c] = empty ? 0 : LLONG_MIN;
        hi[c] = empty ? -1 : LLONG_MAX;
    }
}

__global__ void k_sw_bounds_edges(int64_t E, int32_t C, const int32_t *src, const int32_t *dst,
                                  const int32_t *cluster, const int32_t *level,
                                  const long long *first, const long long *last,
                                  const int64_t *tl, const int64_t *comp, long long *lo,
                                  long long *hi) {
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < E;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int32_t a = src[e], b = dst[e];
        const int32_t ca = cluster[a], cb = cluster[b];
        if (cb >= 0 && cb < C && first[cb] == (((long long)level[b] << 32) | (long long)b))
            atomicMax(&lo[cb], (long long)(tl[a] + comp[a]));
        if (ca >= 0 && ca < C && last[ca] == (((long long)level[a] << 32) | (long long)a))
            atomicMin(&hi[ca], (long long)tl[b]);
    }
}

__global__ void k_sw_bounds_fix(int32_t C, const long long *first, const long long *m,
                                long long *lo, long long *hi) {
    for (int32_t c = blockIdx.x * blockDim.x + threadIdx.x; c < C; c += gridDim.x * blockDim.x) {
        if (first[c] == LLONG_MAX) continue;
        if (lo[c] == LLONG_MIN) lo[c] = 0;
        if (hi[c] == LLONG_MAX) hi[c] = *m;
    }
}

// Eq. 2 communication: edges between a cluster and a node on partition k
__global__ void k_sw_comm(int64_t E, int32_t K, int32_t C, const int32_t *src,
                          const int32_t *dst, const int64_t *cost, const int32_t *cluster,
                          const int32_t *label, unsigned long long *comm) {
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < E;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int32_t a = src[e], b = dst[e];
        const int32_t ca = cluster[a], cb = cluster[b];
        if (ca == cb && ca >= 0) continue;   // inside one cluster
        const unsigned long long w = (unsigned long long)cost[e];
        if (w == 0) continue;
        const int32_t la = label[a], lb = label[b];
        if (ca >= 0 && ca < C && lb >= 0 && lb < K) atomicAdd(&comm[(int64_t)ca * K + lb], w);
        if (cb >= 0 && cb < C && la >= 0 && la < K) atomicAdd(&comm[(int64_t)cb * K + la], w);
    }
}

// first position in [b, e) with s[i] > x (strict) or >= x
template <bool STRICT>
__device__ __forceinline__ int32_t bound(const int64_t *s, int32_t b, int32_t e, int64_t x) {
    while (b < e) {
        const int32_t mid = (int32_t)(((uint32_t)b + (uint32_t)e) >> 1);
        const bool left = STRICT ? (s[mid] <= x) : (s[mid] < x);
        if (left)
            b = mid + 1;
        else
            e = mid;
    }
    return b;
}

// work[c][k]: partition k's weight with tl inside span(c)
__global__ void k_sw_work(int32_t C, int32_t K, const int64_t *lo, const int64_t *hi,
                          const int32_t *seg, const int64_t *s_tl, const int64_t *pre,
                          int64_t *work) {
    const int64_t n = (int64_t)C * K;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int32_t c = (int32_t)(i / K), k = (int32_t)(i - (int64_t)c * K);
        const int64_t a = lo[c], b = hi[c];
        int64_t w = 0;
        if (a <= b) {
            const int32_t s0 = seg[k], s1 = seg[k + 1];
            const int32_t x = bound<false>(s_tl, s0, s1, a);
            const int32_t y = bound<true>(s_tl, x, s1, b);
            w = pre[y] - pre[x];
        }
        work[i] = w;
    }
}

// Work and choice together for K <= 64: a group of G lanes (G = the power of
// two >= K) holds one cluster, lane k its partition k; the group sums the
// communication and picks the Eq. 2 minimum with wave shuffles.
template <int G>
__global__ __launch_bounds__(256) void k_sw_work_decide(
    int32_t C, int32_t K, const int64_t *lo, const int64_t *hi, const int32_t *seg,
    const int64_t *s_tl, const int64_t *pre, const long long *first, const int64_t *comm,
    int64_t *work, int32_t *choice) {
    const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    const int32_t c = (int32_t)(i / G), k = (int32_t)(i % G);
    const bool on = c < C && k < K;
    int64_t w = 0, cm = 0;
    if (on) {
        const int64_t a = lo[c], b = hi[c];
        if (a <= b) {
            const int32_t s0 = seg[k], s1 = seg[k + 1];
            const int32_t x = bound<false>(s_tl, s0, s1, a);
            const int32_t y = bound<true>(s_tl, x, s1, b);
            w = pre[y] - pre[x];
        }
        cm = comm[(int64_t)c * K + k];
        work[(int64_t)c * K + k] = w;
    }
    long long tot = cm;
#pragma unroll
    for (int off = 1; off < G; off <<= 1) tot += __shfl_xor(tot, off, kWave);
    // (cost, -comm, k) lexicographic minimum over the group
    long long cost = on ? (long long)(w + tot - cm) : LLONG_MAX;
    long long neg = on ? -(long long)cm : LLONG_MAX;
    int32_t kk = on ? k : INT32_MAX;
#pragma unroll
    for (int off = 1; off < G; off <<= 1) {
        const long long oc = __shfl_xor(cost, off, kWave), on2 = __shfl_xor(neg, off, kWave);
        const int32_t ok = __shfl_xor(kk, off, kWave);
        if (oc < cost || (oc == cost && (on2 < neg || (on2 == neg && ok < kk)))) {
            cost = oc;
            neg = on2;
            kk = ok;
        }
    }
    if (on && k == 0) choice[c] = first[c] == LLONG_MAX ? -1 : kk;
}

__global__ void k_sw_decide(int32_t C, int32_t K, const long long *first, const int64_t *work,
                            const int64_t *comm, int32_t *choice) {
    for (int32_t c = blockIdx.x * blockDim.x + threadIdx.x; c < C; c += gridDim.x * blockDim.x) {
        if (first[c] == LLONG_MAX) {
            choice[c] = -1;
            continue;
        }
        const int64_t *wr = work + (int64_t)c * K, *cr = comm + (int64_t)c * K;
        int64_t tot = 0;
        for (int32_t k = 0; k < K; k++) tot += cr[k];
        int32_t best = 0;
        int64_t bc = wr[0] + tot - cr[0], bm = cr[0];
        for (int32_t k = 1; k < K; k++) {
            const int64_t cost = wr[k] + tot - cr[k];
            if (cost < bc || (cost == bc && cr[k] > bm)) {
                best = k;
                bc = cost;
                bm = cr[k];
            }
        }
        choice[c] = best;
    }
}

}  // namespace

size_t span_work_scratch_bytes(int32_t V, int32_t C, int32_t K) {
    return SwLayout(V, C, K).total;
}

hipError_t launch_span_work(const Graph &g, const int32_t *label, int32_t K,
                            const int32_t *cluster, int32_t C, const int64_t *tl,
                            int64_t *span_lo, int64_t *span_hi, int64_t *work, int64_t *comm,
                            int32_t *choice, void *scratch, SpanCache *cache, int32_t *err) {
    const int32_t V = g.V;
    const SwLayout L(V, C, K);
    hipStream_t s = g.stream;
    int32_t *ids0 = at<int32_t>(scratch, L.ids0), *ids1 = at<int32_t>(scratch, L.ids1);
    uint64_t *tl_key = at<uint64_t>(scratch, L.tl_key);
    uint64_t *tl_key_out = at<uint64_t>(scratch, L.tl_key_out);
    uint32_t *lab_key = at<uint32_t>(scratch, L.lab_key);
    uint32_t *lab_sorted = at<uint32_t>(scratch, L.lab_sorted);
    int64_t *s_tl = at<int64_t>(scratch, L.s_tl), *wt = at<int64_t>(scratch, L.w);
    int64_t *pre = at<int64_t>(scratch, L.pre);
    int32_t *seg = at<int32_t>(scratch, L.seg);
    int64_t *first = at<int64_t>(scratch, L.first), *last = at<int64_t>(scratch, L.last);
    int64_t *m = at<int64_t>(scratch, L.m);
    void *temp = at<char>(scratch, L.temp);
    hipError_t e;

    if ((e = launch_fill_i64(first, C, LLONG_MAX, s)) != hipSuccess) return e;
    if ((e = launch_fill_i64(last, C, -1, s)) != hipSuccess) return e;
    if ((e = launch_fill_i64(m, 1, LLONG_MIN, s)) != hipSuccess) return e;
    if ((e = launch_fill_i64(pre, 1, 0, s)) != hipSuccess) return e;
    if ((e = launch_fill_i64(comm, (int64_t)C * K, 0, s)) != hipSuccess) return e;
    int pbits = 1;   // partitions 0..K (K: unmapped) fit in pbits bits
    while (pbits < 32 && ((uint64_t)K >> pbits) != 0) pbits++;
    if (V > 0) {
        k_sw_nodes<<<grid_for(V, kBlock, 2048), kBlock, 0, s>>>(
            V, K, C, label, cluster, g.level, tl, g.comp, reinterpret_cast<long long *>(first),
            reinterpret_cast<long long *>(last), reinterpret_cast<long long *>(m), err);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        // the nodes in (tl, id) order, rebuilt only when tl changed; the cache
        // counts as valid again only once every launch of the rebuild is enqueued
        const bool was_valid = cache->valid;
        cache->valid = false;
        if ((e = launch_fill_i32(cache->changed, 1, was_valid ? 0 : 1, s)) != hipSuccess)
            return e;
        if (was_valid) {
            k_sw_tl_cmp<<<grid_for(V, kBlock, 2048), kBlock, 0, s>>>(V, tl, cache->tl,
                                                                     cache->changed);
            if ((e = hipGetLastError()) != hipSuccess) return e;
        }
        k_sw_tl_keys<<<grid_for(V, kBlock), kBlock, 0, s>>>(V, tl, cache->changed, tl_key, ids0,
                                                            cache->tl);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if ((e = sort_pairs_u64(tl_key, tl_key_out, ids0, cache->ids, V, 0, 64, temp, s,
                                cache->changed)) != hipSuccess)
            return e;
        cache->valid = true;
        // split by partition, stably: nodes in (partition, tl, id) order
        k_sw_lab_keys<<<grid_for(V, kBlock), kBlock, 0, s>>>(V, K, label, cache->ids, lab_key);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if ((e = sort_pairs_u32(lab_key, lab_sorted, cache->ids, ids1, V, 0, pbits, temp, s)) !=
            hipSuccess)
            return e;
        k_sw_gather<<<grid_for(V, kBlock), kBlock, 0, s>>>(V, ids1, tl, g.comp, s_tl, wt);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if ((e = inclusive_scan_i64(wt, pre + 1, V, temp, s)) != hipSuccess) return e;
        k_sw_comm<<<grid_for(g.E, kBlock), kBlock, 0, s>>>(
            g.E, K, C, g.e_src, g.e_dst, g.e_cost, cluster, label,
            reinterpret_cast<unsigned long long *>(comm));
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    k_sw_seg<<<grid_for(K + 1, kBlock), kBlock, 0, s>>>(V, K, lab_sorted, seg);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    {
        const long long *fk = reinterpret_cast<const long long *>(first);
        long long *lo = reinterpret_cast<long long *>(span_lo);
        long long *hi = reinterpret_cast<long long *>(span_hi);
        k_sw_bounds_init<<<grid_for(C, kBlock), kBlock, 0, s>>>(C, fk, lo, hi);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if (V > 0 && g.E > 0) {
            k_sw_bounds_edges<<<grid_for(g.E, kBlock), kBlock, 0, s>>>(
                g.E, C, g.e_src, g.e_dst, cluster, g.level, fk,
                reinterpret_cast<const long long *>(last), tl, g.comp, lo, hi);
            if ((e = hipGetLastError()) != hipSuccess) return e;
        }
        k_sw_bounds_fix<<<grid_for(C, kBlock), kBlock, 0, s>>>(
            C, fk, reinterpret_cast<const long long *>(m), lo, hi);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (C == 0) return hipSuccess;
    const long long *fk = reinterpret_cast<const long long *>(first);
    if (K <= 64) {
        int G = 1;
        while (G < K) G <<= 1;
        const unsigned blocks = (unsigned)(((int64_t)C * G + 255) / 256);
        switch (G) {
#define SW_CASE(g_)                                                                              \
    case g_:                                                                                     \
        k_sw_work_decide<g_><<<blocks, 256, 0, s>>>(C, K, span_lo, span_hi, seg, s_tl, pre, fk, \
                                                    comm, work, choice);                         \
        break;
            SW_CASE(1) SW_CASE(2) SW_CASE(4) SW_CASE(8) SW_CASE(16) SW_CASE(32) SW_CASE(64)
#undef SW_CASE
        }
        return hipGetLastError();
    }
    k_sw_work<<<grid_for((int64_t)C * K, kBlock), kBlock, 0, s>>>(C, K, span_lo, span_hi, seg,
                                                                  s_tl, pre, work);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    k_sw_decide<<<grid_for(C, kBlock), kBlock, 0, s>>>(C, K, fk, work, comm, choice);
    return hipGetLastError();
}

}  // namespace pardnn
