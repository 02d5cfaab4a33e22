// sweep.hip -- t-level / b-level sweeps (paper Table 2; Alg. 1
// compute_weighted_levels), for one placement and for a batch of placements.
//
//   tl(v) = max over in-edges (u,v) of tl(u) + comp(u) + c(u,v)     (0 if none)
//   bl(v) = comp(v) + max over out-edges (v,s) of c(v,s) + bl(s)     (comp(v) if none)
//   c(u,v) = 0 when both ends carry the same label, else edge_cost  (Fig. 2
//            caption: communication inside a cluster counts as zero)
//
// Design for gfx950. Dependencies only run from lower to higher levels, so a
// sweep is a chain of L dependent level steps. Each chain is walked by ONE
// persistent workgroup with only workgroup barriers between levels (a grid-wide
// barrier would cost a cross-XCD L2 writeback per level). Inside a level the
// work is EDGE-parallel, not node-parallel: the in-edges (t) or out-edges (b)
// of one level are a single contiguous range of the level-major CSC/CSR, so a
// thread takes one edge, gathers its neighbour's value and label, and folds
// the candidate into an LDS int64 max (ds_max_i64) keyed by the node's slot
// in the level. A second phase walks the level's nodes, reads the LDS
// accumulators and writes the results. High in-degree nodes thus spread over
// many lanes, and a level costs one gather round trip plus two barriers.
//
// Single placement: two workgroups in one launch, one per direction, so t and
// b overlap. Batch: each workgroup owns S placements ("slots") and walks the b
// sweep and then the t sweep for them; the S lanes of one edge read the same
// structure (a broadcast) and S contiguous values of the slice-major arrays,
// and workgroups never wait on one another.
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

__global__ void k_permute_labels(int32_t V, const int32_t *order, const int32_t *placement,
                                 int32_t *lab_lm) {
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < V; i += gridDim.x * blockDim.x)
        lab_lm[i] = placement[order[i]];
}

// ---------------------------------------------------------------------------
// Single placement.
// ---------------------------------------------------------------------------

__device__ void t_sweep_single(const WalkArgs &a, long long *acc) {
    const int tid = threadIdx.x;
    for (int32_t k = 0; k < a.L; k++) {
        const LevelInfo li = a.linfo[k], ln = a.linfo[k + 1];
        for (int32_t lo = li.node_lo; lo < ln.node_lo; lo += kAccNodes) {
            const int32_t hi = min(ln.node_lo, lo + kAccNodes);
            const int32_t ea = lo == li.node_lo ? li.in_e_lo : a.in_off[lo];
            const int32_t eb = hi == ln.node_lo ? ln.in_e_lo : a.in_off[hi];
            for (int32_t e = ea + tid; e < eb; e += kWalkThreads) {
                const int32_t u = a.in_src[e], v = a.in_dst[e];
                const int64_t c = a.in_cost[e];
                const int64_t val = a.ft[u] + (a.lab[u] != a.lab[v] ? c : 0);
                lds_max_i64(&acc[v - lo], val);
            }
            __syncthreads();
            for (int32_t v = lo + tid; v < hi; v += kWalkThreads) {
                const int64_t t = acc[v - lo];
                acc[v - lo] = 0;
                a.ft[v] = t + a.comp_lm[v];
                a.tl_out[a.order[v]] = t;
            }
            __syncthreads();
        }
    }
}

__device__ void b_sweep_single(const WalkArgs &a, long long *acc) {
    const int tid = threadIdx.x;
    for (int32_t k = a.L - 1; k >= 0; k--) {
        const LevelInfo li = a.linfo[k], ln = a.linfo[k + 1];
        for (int32_t lo = li.node_lo; lo < ln.node_lo; lo += kAccNodes) {
            const int32_t hi = min(ln.node_lo, lo + kAccNodes);
            const int32_t ea = lo == li.node_lo ? li.out_e_lo : a.out_off[lo];
            const int32_t eb = hi == ln.node_lo ? ln.out_e_lo : a.out_off[hi];
            for (int32_t e = ea + tid; e < eb; e += kWalkThreads) {
                const int32_t v = a.out_src[e], s = a.out_dst[e];
                const int64_t c = a.out_cost[e];
                const int64_t val = (a.lab[v] != a.lab[s] ? c : 0) + a.blw[s];
                lds_max_i64(&acc[v - lo], val);
            }
            __syncthreads();
            for (int32_t v = lo + tid; v < hi; v += kWalkThreads) {
                const int64_t b = a.comp_lm[v] + acc[v - lo];
                acc[v - lo] = 0;
                a.blw[v] = b;
                a.bl_out[a.order[v]] = b;
            }
            __syncthreads();
        }
    }
    // M = max over v of tl(v) + bl(v) is reached at a node without
    // predecessors (tl = 0 there), i.e. at level 0.
    __shared__ long long wmax[kWalkThreads / kWave];
    long long m = 0;
    const int32_t n0 = a.L > 0 ? a.linfo[1].node_lo : 0;
    for (int32_t v = tid; v < n0; v += kWalkThreads) m = max(m, (long long)a.blw[v]);
    m = wave_max_i64(m);
    if (lane_id() == 0) wmax[wave_id()] = m;
    __syncthreads();
    if (tid == 0) {
        long long r = 0;
        for (int w = 0; w < kWalkThreads / kWave; w++) r = max(r, wmax[w]);
        a.makespan[0] = r;
    }
}

__global__ __launch_bounds__(kWalkThreads) void k_tb_single(WalkArgs a) {
    __shared__ long long acc[kAccNodes];
    for (int i = threadIdx.x; i < kAccNodes; i += kWalkThreads) acc[i] = 0;
    __syncthreads();
    if (blockIdx.x == 0)
        b_sweep_single(a, acc);
    else
        t_sweep_single(a, acc);
}

// ---------------------------------------------------------------------------
// Batch of placements: S slots per workgroup, slice-major scratch.
// ---------------------------------------------------------------------------

template <int S>
__global__ void k_permute_labels_batch(int32_t V, int32_t P, const int32_t *order,
                                       const int32_t *placements, int32_t *lab_w) {
    const int32_t n_slices = (P + S - 1) / S;
    const int64_t total = (int64_t)V * n_slices * S;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        // i runs over (v, slice, slot) with the slot fastest, so reads of
        // one placement row are contiguous.
        const int32_t s = (int32_t)(i % S);
        const int64_t r = i / S;
        const int32_t slice = (int32_t)(r % n_slices);
        const int32_t v = (int32_t)(r / n_slices);
        const int32_t p = slice * S + s;
        const int32_t lab = p < P ? placements[(int64_t)order[v] * P + p] : 0;
        lab_w[((int64_t)slice * V + v) * S + s] = lab;
    }
}

template <int S, int T>
__global__ __launch_bounds__(T) void k_eval_batch(BatchArgs a) {
    constexpr int kAccB = 512;                // nodes per accumulator chunk
    constexpr int kBinsCap = 2048;            // LDS label bins (K * S)
    __shared__ long long acc[kAccB * S];
    __shared__ unsigned long long nacc[kAccB * S];
    __shared__ long long bins[kBinsCap];
    __shared__ long long s_m[S];
    __shared__ int s_start[S], s_next[S], s_len[S];

    const int tid = threadIdx.x;
    const int32_t slice = blockIdx.x;
    const int32_t p0 = slice * S;
    const int64_t wbase = (int64_t)slice * a.V * S;
    const int32_t *lab = a.lab_w + wbase;
    int64_t *ft = a.ft_w + wbase;
    int64_t *bl = a.bl_w + wbase;
    int32_t *nx = a.nx_w + wbase;
    const bool want_path = a.path != nullptr;
    const bool lds_bins = a.K > 0 && a.K * S <= kBinsCap;

    for (int i = tid; i < kAccB * S; i += T) {
        acc[i] = 0;
        nacc[i] = ~0ull;
    }
    if (lds_bins)
        for (int i = tid; i < a.K * S; i += T) bins[i] = 0;
    if (tid < S) {
        s_m[tid] = 0;
        s_start[tid] = INT32_MAX;
        s_len[tid] = 0;
    }
    __syncthreads();

    // ---- b sweep, levels L-1 .. 0 ----
    for (int32_t k = a.L - 1; k >= 0; k--) {
        const LevelInfo li = a.linfo[k], ln = a.linfo[k + 1];
        for (int32_t lo = li.node_lo; lo < ln.node_lo; lo += kAccB) {
            const int32_t hi = min(ln.node_lo, lo + kAccB);
            const int32_t ea = lo == li.node_lo ? li.out_e_lo : a.out_off[lo];
            const int32_t eb = hi == ln.node_lo ? ln.out_e_lo : a.out_off[hi];
            const int32_t ne = (eb - ea) * S;
            for (int32_t i = tid; i < ne; i += T) {
                const int32_t e = ea + i / S, s = i % S;
                const int32_t v = a.out_src[e], sn = a.out_dst[e];
                const int64_t c = a.out_cost[e];
                const int64_t val =
                    (lab[(int64_t)v * S + s] != lab[(int64_t)sn * S + s] ? c : 0) +
                    bl[(int64_t)sn * S + s];
                lds_max_i64(&acc[(v - lo) * S + s], val);
            }
            __syncthreads();
            if (want_path) {
                // smallest original id among the successors reaching the max
                for (int32_t i = tid; i < ne; i += T) {
                    const int32_t e = ea + i / S, s = i % S;
                    const int32_t v = a.out_src[e], sn = a.out_dst[e];
                    const int64_t c = a.out_cost[e];
                    const int64_t val =
                        (lab[(int64_t)v * S + s] != lab[(int64_t)sn * S + s] ? c : 0) +
                        bl[(int64_t)sn * S + s];
                    if (val == acc[(v - lo) * S + s]) {
                        const unsigned long long key =
                            ((unsigned long long)(uint32_t)a.out_dst_orig[e] << 32) |
                            (uint32_t)sn;
                        lds_min_u64(&nacc[(v - lo) * S + s], key);
                    }
                }
                __syncthreads();
            }
            const int32_t nn = (hi - lo) * S;
            for (int32_t i = tid; i < nn; i += T) {
                const int32_t v = lo + i / S, s = i % S;
                const int32_t slot = (v - lo) * S + s;
                const int64_t b = a.comp_lm[v] + acc[slot];
                acc[slot] = 0;
                bl[(int64_t)v * S + s] = b;
                if (want_path) {
                    const unsigned long long key = nacc[slot];
                    nacc[slot] = ~0ull;
                    nx[(int64_t)v * S + s] = key == ~0ull ? -1 : (int32_t)(key & 0xffffffffull);
                }
                if (p0 + s < a.P) a.bl_out[(int64_t)a.order[v] * a.P + p0 + s] = b;
            }
            __syncthreads();
        }
    }

    // ---- makespan and path start per slot (level 0: tl = 0 there) ----
    const int32_t n0 = a.L > 0 ? a.linfo[1].node_lo : 0;
    for (int32_t i = tid; i < n0 * S; i += T) {
        const int32_t v = i / S, s = i % S;
        lds_max_i64(&s_m[s], bl[(int64_t)v * S + s]);
    }
    __syncthreads();
    for (int32_t i = tid; i < n0 * S; i += T) {
        const int32_t v = i / S, s = i % S;
        // level 0 is sorted by original id, so the smallest lm index is the
        // smallest original id
        if (bl[(int64_t)v * S + s] == s_m[s]) lds_min_i32(&s_start[s], v);
    }
    __syncthreads();
    if (tid < S) {
        s_next[tid] = s_start[tid] == INT32_MAX ? -1 : s_start[tid];
        if (p0 + tid < a.P) a.makespan[p0 + tid] = s_m[tid];
    }
    __syncthreads();

    // ---- t sweep, levels 0 .. L-1, with critical flags, path and label sums ----
    for (int32_t k = 0; k < a.L; k++) {
        const LevelInfo li = a.linfo[k], ln = a.linfo[k + 1];
        for (int32_t lo = li.node_lo; lo < ln.node_lo; lo += kAccB) {
            const int32_t hi = min(ln.node_lo, lo + kAccB);
            const int32_t ea = lo == li.node_lo ? li.in_e_lo : a.in_off[lo];
            const int32_t eb = hi == ln.node_lo ? ln.in_e_lo : a.in_off[hi];
            const int32_t ne = (eb - ea) * S;
            for (int32_t i = tid; i < ne; i += T) {
                const int32_t e = ea + i / S, s = i % S;
                const int32_t u = a.in_src[e], v = a.in_dst[e];
                const int64_t c = a.in_cost[e];
                const int64_t val =
                    ft[(int64_t)u * S + s] +
                    (lab[(int64_t)u * S + s] != lab[(int64_t)v * S + s] ? c : 0);
                lds_max_i64(&acc[(v - lo) * S + s], val);
            }
            __syncthreads();
            const int32_t nn = (hi - lo) * S;
            for (int32_t i = tid; i < nn; i += T) {
                const int32_t v = lo + i / S, s = i % S;
                const int32_t slot = (v - lo) * S + s;
                const int64_t t = acc[slot];
                acc[slot] = 0;
                ft[(int64_t)v * S + s] = t + a.comp_lm[v];
                const int32_t p = p0 + s;
                if (p >= a.P) continue;
                const int32_t ov = a.order[v];
                a.tl_out[(int64_t)ov * a.P + p] = t;
                if (a.crit_out)
                    a.crit_out[(int64_t)ov * a.P + p] =
                        (uint8_t)(t + bl[(int64_t)v * S + s] == s_m[s]);
                if (a.K > 0) {
                    const int32_t l = lab[(int64_t)v * S + s];
                    if (l < 0 || l >= a.K) {
                        atomicOr(a.err, 1);
                    } else if (lds_bins) {
                        lds_add_i64(&bins[l * S + s], a.mem_lm[v]);
                    } else {
                        atomicAdd((unsigned long long *)&a.label_mem[(int64_t)p * a.K + l],
                                  (unsigned long long)a.mem_lm[v]);
                    }
                }
                if (want_path && v == s_next[s]) {
                    // the successor lies on a later level, so no other thread
                    // of this level can match the updated value
                    a.path[(int64_t)p * a.path_stride + s_len[s]] = ov;
                    s_len[s] = s_len[s] + 1;
                    s_next[s] = nx[(int64_t)v * S + s];
                }
            }
            __syncthreads();
        }
    }
    if (tid < S && p0 + tid < a.P && want_path) a.path_len[p0 + tid] = s_len[tid];
    if (lds_bins) {
        for (int i = tid; i < a.K * S; i += T) {
            const int l = i / S, s = i % S;
            if (p0 + s < a.P) a.label_mem[(int64_t)(p0 + s) * a.K + l] = bins[i];
        }
    }
}

constexpr int kBatchSlots = 2;
constexpr int kBatchThreads = 256;

}  // namespace

hipError_t launch_permute_labels(const Graph &g, const int32_t *placement, int32_t *lab_lm) {
    if (g.V == 0) return hipSuccess;
    k_permute_labels<<<grid_for(g.V, kBlock), kBlock, 0, g.stream>>>(g.V, g.order, placement,
                                                                      lab_lm);
    return hipGetLastError();
}

hipError_t launch_tb_single(const WalkArgs &a, hipStream_t s) {
    k_tb_single<<<2, kWalkThreads, 0, s>>>(a);
    return hipGetLastError();
}

int batch_slots() { return kBatchSlots; }

hipError_t launch_permute_labels_batch(const Graph &g, const int32_t *placements, int32_t P,
                                       int32_t S, int32_t *lab_w) {
    if (S != kBatchSlots) return hipErrorInvalidValue;
    const int64_t n_slices = (P + S - 1) / S;
    const int64_t total = (int64_t)g.V * n_slices * S;
    if (total == 0) return hipSuccess;
    k_permute_labels_batch<kBatchSlots><<<grid_for(total, kBlock), kBlock, 0, g.stream>>>(
        g.V, P, g.order, placements, lab_w);
    return hipGetLastError();
}

hipError_t launch_eval_batch(const BatchArgs &a, int32_t S, hipStream_t s) {
    if (S != kBatchSlots) return hipErrorInvalidValue;
    const int32_t n_slices = (a.P + S - 1) / S;
    if (n_slices == 0) return hipSuccess;
    k_eval_batch<kBatchSlots, kBatchThreads><<<n_slices, kBatchThreads, 0, s>>>(a);
    return hipGetLastError();
}

}  // namespace pardnn
