// clusters.hip -- cluster criticality of the mapping stage (paper Sec. 3.1.2).
//
// After slicing, the criticality of a linear cluster is the length of the
// longest source-to-sink path through it when communication inside every
// cluster counts as zero; the clusters are then taken in non-increasing order
// of criticality. With the cluster ids as labels, the weighted levels w(n) =
// tl(n) + bl(n) of that evaluation give
//   criticality(c) = max over the nodes n of cluster c of w(n)   (-1: no node)
// and the order sorts clusters by (criticality descending, id ascending).
//
// Design for gfx950: the weighted levels come from the single-placement
// sweep; the per-cluster maximum is one pass of 64-bit atomic maxima (cluster
// ids are arbitrary, up to one per node); the order is a stable radix sort of
// the keys bound - criticality (ascending, so criticality descending) over the
// ids given ascending, bound being the ingest bound on every path length.
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

__global__ void k_cluster_max(int32_t V, int32_t n_clusters, const int32_t *cluster,
                              const int64_t *tl, const int64_t *bl, long long *crit,
                              int32_t *err) {
    for (int32_t v = blockIdx.x * blockDim.x + threadIdx.x; v < V; v += gridDim.x * blockDim.x) {
        const int32_t c = cluster[v];
        if ((uint32_t)c >= (uint32_t)n_clusters) {
            atomicOr(err, 1);
            continue;
        }
        atomicMax(&crit[c], (long long)(tl[v] + bl[v]));
    }
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

// Scratch of the sort: keys in and out (uint64[n] each), ids int32[n], then
// the radix sort's own space. Returns the bytes needed for n clusters.
size_t cluster_sort_bytes(int32_t n) {
    return 3 * (((size_t)n * 8 + 255) / 256 * 256) + sort_pairs_scratch_bytes(n, 8);
}

namespace {

// key = bound - criticality: criticality in [-1, bound] gives keys in
// [0, bound + 1], smaller for more critical clusters
__global__ void k_cl_keys(int32_t C, uint64_t bound, const int64_t *crit, uint64_t *key) {
    for (int32_t c = blockIdx.x * blockDim.x + threadIdx.x; c < C; c += gridDim.x * blockDim.x)
        key[c] = bound - (uint64_t)crit[c];
}

}  // namespace

hipError_t launch_cluster_criticality(const Graph &g, const int32_t *cluster, int32_t n_clusters,
                                      const int64_t *tl, const int64_t *bl, int64_t *crit,
                                      int32_t *order, void *scratch, size_t scratch_bytes,
                                      int32_t *err) {
    hipError_t e = launch_fill_i64(crit, n_clusters, -1, g.stream);
    if (e != hipSuccess) return e;
    if (g.V > 0) {
        k_cluster_max<<<grid_for(g.V, kBlock), kBlock, 0, g.stream>>>(
            g.V, n_clusters, cluster, tl, bl, reinterpret_cast<long long *>(crit), err);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (scratch_bytes < cluster_sort_bytes(n_clusters)) return hipErrorInvalidValue;
    const size_t seg = ((size_t)n_clusters * 8 + 255) / 256 * 256;
    uint64_t *keys_in = reinterpret_cast<uint64_t *>(scratch);
    uint64_t *keys_out = reinterpret_cast<uint64_t *>(reinterpret_cast<char *>(scratch) + seg);
    int32_t *ids = reinterpret_cast<int32_t *>(reinterpret_cast<char *>(scratch) + 2 * seg);
    void *temp = reinterpret_cast<char *>(scratch) + 3 * seg;
    const uint64_t bound = (uint64_t)g.weight_bound;
    int bits = 1;
    while (bits < 64 && ((bound + 1) >> bits) != 0) bits++;
    k_cl_keys<<<grid_for(n_clusters, kBlock), kBlock, 0, g.stream>>>(n_clusters, bound, crit,
                                                                     keys_in);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = launch_iota_i32(ids, n_clusters, g.stream)) != hipSuccess) return e;
    return sort_pairs_u64(keys_in, keys_out, ids, order, n_clusters, 0, bits, temp, g.stream);
}

}  // namespace pardnn
