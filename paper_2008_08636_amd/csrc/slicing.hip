// slicing.hip -- the primary clusters of graph slicing (paper Alg. 1, Sec.
// 3.1.1): K rounds of [weighted levels of the remaining graph -> its heaviest
// (critical) path -> remove that path's nodes and their edges].
//
// Before any placement every edge carries its communication cost, so the
// rounds evaluate with pairwise distinct labels. Removal is expressed through
// the node weights the sweep reads: a removed node weighs -B, B larger than
// every path of the graph, so any candidate through it is negative and loses
// to the empty maximum 0 -- exactly as if the node and its edges were gone.
// The path then starts at the smallest-id critical node that has no remaining
// predecessor (a source of the remaining graph) and follows the tight
// successors, which are never removed nodes.
//
// Design for gfx950: a round is one single-placement sweep (latency-bound,
// one chain per direction), one tight-successor pass and a one-workgroup
// chase, all enqueued without host synchronisation; only the removal and the
// start search are added here, each a data-parallel pass.
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

__global__ void k_slice_init(int32_t V, const NodeRec16 *node_rec, const int64_t *comp_lm,
                             NodeRec16 *node_rec_s, int64_t *comp_lm_s, uint8_t *alive_lm,
                             int32_t *primary) {
    for (int32_t v = blockIdx.x * blockDim.x + threadIdx.x; v < V; v += gridDim.x * blockDim.x) {
        node_rec_s[v] = node_rec[v];
        comp_lm_s[v] = comp_lm[v];
        alive_lm[v] = 1;
        primary[v] = -1;
    }
}

// M of the remaining graph: the largest tl + bl over its nodes (0 when none
// remains). A source of the remaining graph may sit at any level, so this is
// not the sweep's level-0 maximum.
__global__ void k_slice_max(int32_t V, const int32_t *order, const uint8_t *alive_lm,
                            const int64_t *tl, const int64_t *bl, int64_t *makespan) {
    long long m = 0;
    for (int32_t v = blockIdx.x * blockDim.x + threadIdx.x; v < V; v += gridDim.x * blockDim.x) {
        if (!alive_lm[v]) continue;
        const int32_t o = order[v];
        const long long w = tl[o] + bl[o];
        m = w > m ? w : m;
    }
    m = wave_max_i64(m);
    if ((threadIdx.x & (kWave - 1)) == 0 && m > 0) atomicMax((long long *)makespan, m);
}

// smallest original id among the critical nodes without a remaining
// predecessor (level-major CSC of in-edges)
__global__ void k_slice_start(int32_t V, const int32_t *order, const int32_t *in_off,
                              const int32_t *in_src, const uint8_t *alive_lm,
                              const uint8_t *crit_lm, int32_t *start) {
    for (int32_t v = blockIdx.x * blockDim.x + threadIdx.x; v < V; v += gridDim.x * blockDim.x) {
        if (!alive_lm[v] || !crit_lm[v]) continue;
        bool source = true;
        for (int32_t j = in_off[v]; j < in_off[v + 1] && source; j++) source = !alive_lm[in_src[j]];
        if (source) atomicMin(start, order[v]);
    }
}

// the round's path leaves the graph: its nodes weigh -B from now on
__global__ void k_slice_remove(int32_t round, const int32_t *path, const int32_t *path_len,
                               const int32_t *rank, int64_t big, NodeRec16 *node_rec_s,
                               int64_t *comp_lm_s, uint8_t *alive_lm, int32_t *primary) {
    const int32_t n = *path_len;
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
        const int32_t o = path[i], v = rank[o];
        node_rec_s[v].comp = -big;
        comp_lm_s[v] = -big;
        alive_lm[v] = 0;
        primary[o] = round;
    }
}

}  // namespace

hipError_t launch_slice_init(const Graph &g, NodeRec16 *node_rec_s, int64_t *comp_lm_s,
                             uint8_t *alive_lm, int32_t *primary) {
    if (g.V == 0) return hipSuccess;
    k_slice_init<<<grid_for(g.V, kBlock), kBlock, 0, g.stream>>>(g.V, g.node_rec, g.comp_lm,
                                                                 node_rec_s, comp_lm_s, alive_lm,
                                                                 primary);
    return hipGetLastError();
}

hipError_t launch_slice_makespan(const Graph &g, const uint8_t *alive_lm, const int64_t *tl,
                                const int64_t *bl, int64_t *makespan) {
    hipError_t e = launch_fill_i64(makespan, 1, 0, g.stream);
    if (e != hipSuccess || g.V == 0) return e;
    k_slice_max<<<grid_for(g.V, kBlock, 1024), kBlock, 0, g.stream>>>(g.V, g.order, alive_lm, tl,
                                                                     bl, makespan);
    return hipGetLastError();
}

hipError_t launch_slice_start(const Graph &g, const uint8_t *alive_lm, int32_t *start) {
    hipError_t e = launch_fill_i32(start, 1, INT32_MAX, g.stream);
    if (e != hipSuccess || g.V == 0) return e;
    k_slice_start<<<grid_for(g.V, kBlock), kBlock, 0, g.stream>>>(g.V, g.order, g.in_off,
                                                                  g.in_src, alive_lm, g.crit_lm,
                                                                  start);
    return hipGetLastError();
}

hipError_t launch_slice_remove(const Graph &g, int32_t round, const int32_t *path,
                               const int32_t *path_len, int64_t big, NodeRec16 *node_rec_s,
                               int64_t *comp_lm_s, uint8_t *alive_lm, int32_t *primary) {
    k_slice_remove<<<grid_for(g.V, kBlock, 1024), kBlock, 0, g.stream>>>(
        round, path, path_len, g.rank, big, node_rec_s, comp_lm_s, alive_lm, primary);
    return hipGetLastError();
}

}  // namespace pardnn
