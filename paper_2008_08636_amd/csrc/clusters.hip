// clusters.hip -- cluster criticality of the mapping stage (paper Sec. 3.1.2).
//
// After slicing, the criticality of a linear cluster (a path) is the length of
// the longest source-to-sink path that runs along the whole cluster when
// communication inside every cluster counts as zero; the clusters are then
// taken in non-increasing order of criticality. With the cluster ids as
// labels, the weighted levels tl / bl of that evaluation give
//   criticality(c) = tl(first) + sum of comp over c + bl(last) - comp(last)
// where first / last are the cluster's nodes of smallest / largest (level,
// id); a cluster whose nodes in that order are not joined by an edge from each
// to the next is no path and gets -1, as does a cluster without nodes. The
// order sorts clusters by (criticality descending, id ascending).
//
// Design for gfx950: the weighted levels come from the single-placement
// sweep. The nodes, given in level-major order, are radix-sorted stably by
// cluster id, so that each cluster's members lie together in path order; an
// edge-parallel pass marks the nodes that have an edge to the next member
// (hub nodes with thousands of edges cost no serial loop), a pass over the
// sorted members counts those links and sums the computation weights per
// cluster (one atomic per wave when the wave's members share a cluster), and
// one thread per cluster applies the formula. The order is a stable radix
// sort of the keys bound - criticality (ascending, so criticality descending)
// over the ids given ascending, bound being the ingest bound on every path
// length.
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

__global__ void k_cl_count(int32_t V, int32_t C, const int32_t *cluster, int32_t *count) {
    for (int32_t v = blockIdx.x * blockDim.x + threadIdx.x; v < V; v += gridDim.x * blockDim.x) {
        const int32_t c = cluster[v];
        if ((uint32_t)c < (uint32_t)C) atomicAdd(&count[c], 1);
    }
}

__global__ void k_cl_multi(int32_t C, const int32_t *count, int32_t *flag) {
    for (int32_t c = blockIdx.x * blockDim.x + threadIdx.x; c < C; c += gridDim.x * blockDim.x)
        flag[c] = count[c] >= 2 ? 1 : 0;
}

// a node of a cluster with two or more nodes takes L + the cluster's rank
// among those; a node alone in its cluster takes its level
__global__ void k_cl_labels(int32_t V, int32_t C, int32_t L, const int32_t *cluster,
                            const int32_t *count, const int32_t *rank, const int32_t *level,
                            int32_t *lab) {
    for (int32_t v = blockIdx.x * blockDim.x + threadIdx.x; v < V; v += gridDim.x * blockDim.x) {
        const int32_t c = cluster[v];
        const bool multi = (uint32_t)c < (uint32_t)C && count[c] >= 2;
        lab[v] = multi ? L + rank[c] : level[v];
    }
}

}  // namespace

// Labels with the same equality on every edge as the cluster ids, drawn from
// few values: communication matters only across an edge, and an edge always
// joins two levels, so a node alone in its cluster can carry its level; the
// clusters with two or more nodes take the values L, L + 1, ... in id order.
// Scratch: count, flag int32[C], rank int32[C + 1], the scan's space; lab is
// int32[V]. rank[C] receives the number of clusters with two or more nodes.
size_t cluster_relabel_bytes(int32_t V, int32_t C) {
    const size_t n = 3 * (size_t)C + 1 + scan_workspace_elems(C) + (size_t)V;
    return (n * 4 + 255) / 256 * 256;
}

hipError_t launch_cluster_relabel(const Graph &g, const int32_t *cluster, int32_t C,
                                  int32_t *scratch, int32_t **lab, int32_t **n_multi) {
    int32_t *count = scratch, *flag = count + C, *rank = flag + C;
    int32_t *ws = rank + C + 1;
    *lab = ws + scan_workspace_elems(C);
    *n_multi = rank + C;
    hipError_t e = launch_fill_i32(count, C, 0, g.stream);
    if (e != hipSuccess) return e;
    if (g.V > 0) {
        k_cl_count<<<grid_for(g.V, kBlock), kBlock, 0, g.stream>>>(g.V, C, cluster, count);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    k_cl_multi<<<grid_for(C, kBlock), kBlock, 0, g.stream>>>(C, count, flag);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = launch_exclusive_scan(flag, rank, C, ws, g.stream)) != hipSuccess) return e;
    if (g.V > 0) {
        k_cl_labels<<<grid_for(g.V, kBlock), kBlock, 0, g.stream>>>(g.V, C, g.L, cluster, count,
                                                                    rank, g.level, *lab);
        e = hipGetLastError();
    }
    return e;
}

namespace {

inline size_t al256(size_t b) { return (b + 255) / 256 * 256; }

// Scratch of the criticality pass for V nodes and C clusters.
struct ClLayout {
    size_t keys_in, keys_out, vals_in, vals_out, nxt, lk, fp, lp, nlink, sum, ck_in, ck_out,
        ids, temp, total;
    ClLayout(int32_t V, int32_t C) {
        size_t o = 0;
        auto take = [&](size_t bytes) {
            const size_t at = o;
            o += al256(bytes);
            return at;
        };
        keys_in = take((size_t)V * 4);
        keys_out = take((size_t)V * 4);
        vals_in = take((size_t)V * 4);
        vals_out = take((size_t)V * 4);
        nxt = take((size_t)V * 4);
        lk = take((size_t)V * 4);
        fp = take((size_t)C * 4);
        lp = take((size_t)C * 4);
        nlink = take((size_t)C * 4);
        sum = take((size_t)C * 8);
        ck_in = take((size_t)C * 8);
        ck_out = take((size_t)C * 8);
        ids = take((size_t)C * 4);
        temp = take(std::max(sort_pairs_scratch_bytes(V, 4), sort_pairs_scratch_bytes(C, 8)));
        total = o;
    }
};

template <class T>
T *at_off(void *base, size_t off) {
    return reinterpret_cast<T *>(reinterpret_cast<char *>(base) + off);
}

// key = cluster of level-major node v (C for an id out of range, flagged),
// value = v: sorted stably by key, each cluster's members come out in
// level-major order
__global__ void k_cl_node_keys(int32_t V, int32_t C, const int32_t *order, const int32_t *cluster,
                               uint32_t *key, int32_t *val, int32_t *lk, int32_t *err) {
    for (int32_t v = blockIdx.x * blockDim.x + threadIdx.x; v < V; v += gridDim.x * blockDim.x) {
        const int32_t c = cluster[order[v]];
        const bool bad = (uint32_t)c >= (uint32_t)C;
        if (bad) atomicOr(err, 1);
        key[v] = bad ? (uint32_t)C : (uint32_t)c;
        val[v] = v;
        lk[v] = 0;
    }
}

// per sorted position i: the member after it (nxt), the cluster's first and
// last positions, and its computation weight into the cluster's sum
__global__ void k_cl_segments(int32_t V, int32_t C, const uint32_t *key, const int32_t *val,
                              const int64_t *comp_lm, int32_t *nxt, int32_t *fp, int32_t *lp,
                              unsigned long long *sum) {
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < V; i += gridDim.x * blockDim.x) {
        const uint32_t c = key[i];
        const int32_t v = val[i];
        const bool more = i + 1 < V && key[i + 1] == c;
        nxt[v] = more ? val[i + 1] : -1;
        if (c >= (uint32_t)C) continue;
        if (i == 0 || key[i - 1] != c) fp[c] = i;
        if (!more) lp[c] = i;
        atomicAdd(&sum[c], (unsigned long long)comp_lm[v]);
    }
}

// edge-parallel over the level-major out-edges: u links to its next member
__global__ void k_cl_link(int64_t E, const int32_t *out_src, const int32_t *out_dst,
                          const int32_t *nxt, int32_t *lk) {
    for (int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; j < E;
         j += (int64_t)gridDim.x * blockDim.x) {
        const int32_t u = out_src[j];
        if (nxt[u] == out_dst[j]) lk[u] = 1;
    }
}

// links per cluster over the sorted members: one atomic per wave when all of
// its lanes hold members of one cluster, else one per linked member
__global__ void k_cl_count_links(int32_t V, int32_t C, const uint32_t *key, const int32_t *val,
                                 const int32_t *lk, int32_t *nlink) {
    const int32_t stride = gridDim.x * blockDim.x;
    for (int32_t i0 = blockIdx.x * blockDim.x; i0 < V; i0 += stride) {
        const int32_t i = i0 + threadIdx.x;
        const bool in = i < V;
        const uint32_t c = in ? key[i] : 0xffffffffu;
        const bool linked = in && c < (uint32_t)C && lk[val[i]] != 0;
        const uint32_t c0 = __shfl(c, 0, kWave);
        if (__ballot(c != c0) == 0ull) {
            const int n = __popcll(__ballot(linked));
            if (lane_id() == 0 && n > 0) atomicAdd(&nlink[c0], n);
        } else if (linked) {
            atomicAdd(&nlink[c], 1);
        }
    }
}

__global__ void k_cl_final(int32_t C, const int32_t *fp, const int32_t *lp, const int32_t *nlink,
                           const long long *sum, const int32_t *val, const int32_t *order,
                           const int64_t *comp_lm, const int64_t *tl, const int64_t *bl,
                           int64_t *crit) {
    for (int32_t c = blockIdx.x * blockDim.x + threadIdx.x; c < C; c += gridDim.x * blockDim.x) {
        const int32_t a = fp[c];
        int64_t x = -1;
        if (a >= 0 && nlink[c] == lp[c] - a) {
            const int32_t first = val[a], last = val[lp[c]];
            x = tl[order[first]] + sum[c] + bl[order[last]] - comp_lm[last];
        }
        crit[c] = x;
    }
}

// key = bound - criticality: criticality in [-1, bound] gives keys in
// [0, bound + 1], smaller for more critical clusters
__global__ void k_cl_keys(int32_t C, uint64_t bound, const int64_t *crit, uint64_t *key) {
    for (int32_t c = blockIdx.x * blockDim.x + threadIdx.x; c < C; c += gridDim.x * blockDim.x)
        key[c] = bound - (uint64_t)crit[c];
}

}  // namespace

size_t cluster_sort_bytes(int32_t V, int32_t n) { return ClLayout(V, n).total; }

hipError_t launch_cluster_criticality(const Graph &g, const int32_t *cluster, int32_t C,
                                      const int64_t *tl, const int64_t *bl, int64_t *crit,
                                      int32_t *order, void *scratch, size_t scratch_bytes,
                                      int32_t *err) {
    const int32_t V = g.V;
    const ClLayout L(V, C);
    if (scratch_bytes < L.total) return hipErrorInvalidValue;
    hipStream_t s = g.stream;
    uint32_t *keys_in = at_off<uint32_t>(scratch, L.keys_in);
    uint32_t *keys_out = at_off<uint32_t>(scratch, L.keys_out);
    int32_t *vals_in = at_off<int32_t>(scratch, L.vals_in);
    int32_t *vals_out = at_off<int32_t>(scratch, L.vals_out);
    int32_t *nxt = at_off<int32_t>(scratch, L.nxt), *lk = at_off<int32_t>(scratch, L.lk);
    int32_t *fp = at_off<int32_t>(scratch, L.fp), *lp = at_off<int32_t>(scratch, L.lp);
    int32_t *nlink = at_off<int32_t>(scratch, L.nlink);
    int64_t *sum = at_off<int64_t>(scratch, L.sum);
    uint64_t *ck_in = at_off<uint64_t>(scratch, L.ck_in);
    uint64_t *ck_out = at_off<uint64_t>(scratch, L.ck_out);
    int32_t *ids = at_off<int32_t>(scratch, L.ids);
    void *temp = at_off<char>(scratch, L.temp);
    hipError_t e;
    if ((e = launch_fill_i32(fp, C, -1, s)) != hipSuccess) return e;
    if ((e = launch_fill_i32(lp, C, -1, s)) != hipSuccess) return e;
    if ((e = launch_fill_i32(nlink, C, 0, s)) != hipSuccess) return e;
    if ((e = launch_fill_i64(sum, C, 0, s)) != hipSuccess) return e;
    if (V > 0) {
        k_cl_node_keys<<<grid_for(V, kBlock), kBlock, 0, s>>>(V, C, g.order, cluster, keys_in,
                                                              vals_in, lk, err);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        int bits = 1;
        while (bits < 32 && ((uint32_t)C >> bits) != 0) bits++;
        if ((e = sort_pairs_u32(keys_in, keys_out, vals_in, vals_out, V, 0, bits, temp, s)) !=
            hipSuccess)
            return e;
        k_cl_segments<<<grid_for(V, kBlock), kBlock, 0, s>>>(
            V, C, keys_out, vals_out, g.comp_lm, nxt, fp, lp,
            reinterpret_cast<unsigned long long *>(sum));
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if (g.E > 0) {
            k_cl_link<<<grid_for(g.E, kBlock), kBlock, 0, s>>>(g.E, g.out_src, g.out_dst, nxt,
                                                               lk);
            if ((e = hipGetLastError()) != hipSuccess) return e;
        }
        k_cl_count_links<<<grid_for(V, kBlock), kBlock, 0, s>>>(V, C, keys_out, vals_out, lk,
                                                                nlink);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    k_cl_final<<<grid_for(C, kBlock), kBlock, 0, s>>>(
        C, fp, lp, nlink, reinterpret_cast<const long long *>(sum), vals_out, g.order,
        g.comp_lm, tl, bl, crit);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const uint64_t bound = (uint64_t)g.weight_bound;
    int bits = 1;
    while (bits < 64 && ((bound + 1) >> bits) != 0) bits++;
    k_cl_keys<<<grid_for(C, kBlock), kBlock, 0, s>>>(C, bound, crit, ck_in);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = launch_iota_i32(ids, C, s)) != hipSuccess) return e;
    return sort_pairs_u64(ck_in, ck_out, ids, order, C, 0, bits, temp, s);
}

}  // namespace pardnn
