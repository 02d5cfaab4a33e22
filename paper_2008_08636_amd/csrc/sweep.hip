// sweep.hip -- t-level / b-level sweeps (paper Table 2; Alg. 1
// compute_weighted_levels), for one placement and for a batch of placements,
// plus the batched critical flags and critical-path walk.
//
//   tl(v) = max over in-edges (u,v) of tl(u) + comp(u) + c(u,v)     (0 if none)
//   bl(v) = comp(v) + max over out-edges (v,s) of c(v,s) + bl(s)     (comp(v) if none)
//   c(u,v) = 0 when both ends carry the same label, else edge_cost  (Fig. 2
//            caption: communication inside a cluster counts as zero)
//
// Design for gfx950. Dependencies only run from lower to higher levels, so a
// sweep is a chain of L dependent level steps. Each chain is walked by ONE
// persistent workgroup with only workgroup barriers between levels (a grid-wide
// barrier would cost a cross-XCD L2 writeback per level). The t chain and the
// b chain of a placement are independent, so they run in different
// workgroups at the same time.
//
// Inside a level the work is EDGE-parallel: the in-edges (t) or out-edges (b)
// of one level are one contiguous range of the level-major CSC/CSR, so a thread
// takes one (edge, placement) task, gathers its neighbour's {value, label}
// pair with a single 16-byte load, and folds the candidate into an LDS int64
// max (ds_max_i64) keyed by the node's slot in the level. A node phase then
// reads the accumulators and writes the results. Everything a level needs
// except the neighbour values -- its edge records, its nodes' costs, ids and
// labels -- depends on the structure only, so it is loaded during the
// previous level (registers, and LDS for the labels): a level step costs one
// gather round trip plus LDS work and barriers. Levels wider than the LDS
// accumulators are processed in chunks without prefetch.
//
// Batch: a workgroup owns S placements ("slots") of one direction; the S
// lanes of one edge read the same structure (a broadcast) and S adjacent
// {value, label} pairs of the slice-major workspace.
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

// Lanes of one placement slice: labels gathered into the slice-major layout
// [slice][V][S] through an LDS tile, so that both the reads of the caller's
// placement rows and the writes are contiguous.
template <int S>
__global__ __launch_bounds__(256) void k_permute_labels(int32_t V, int32_t P,
                                                        const int32_t *order,
                                                        const int32_t *placements,
                                                        int32_t *lab_w) {
    constexpr int TV = 64, TP = 64;  // tile: 64 nodes x 64 placements
    __shared__ int32_t tile[TV][TP + 1];
    const int32_t n_slices = (P + S - 1) / S;
    const int32_t v0 = blockIdx.x * TV;
    const int32_t q0 = blockIdx.y * TP;  // first placement of the tile
    const int tx = threadIdx.x & (TP - 1), ty = threadIdx.x / TP;
    for (int r = ty; r < TV; r += 256 / TP) {
        const int32_t v = v0 + r, p = q0 + tx;
        int32_t x = 0;
        if (v < V && p < P) x = placements[(int64_t)order[v] * P + p];
        tile[r][tx] = x;
    }
    __syncthreads();
    // write: for each slice in the tile, TV nodes x S slots, contiguous
    const int32_t sl0 = q0 / S;
    const int n_sl = min(TP / S, n_slices - sl0);
    for (int i = threadIdx.x; i < n_sl * TV * S; i += 256) {
        const int sl = i / (TV * S);
        const int rem = i % (TV * S);
        const int r = rem / S, s = rem % S;
        const int32_t v = v0 + r;
        if (v < V) lab_w[((int64_t)(sl0 + sl) * V + v) * S + s] = tile[r][sl * S + s];
    }
}

struct alignas(16) Pair {
    int64_t val;
    int64_t lab;
};

// Storage of one node's {value, label} in the sweep workspace. Packed: one
// int64 key (value << lb) | label, valid when every label fits in lb bits and
// every value in 63 - lb bits (checked by the host); otherwise a 16-byte pair.
template <bool PACKED>
struct Elem;
template <>
struct Elem<true> {
    using T = int64_t;
    __device__ static int64_t val(T e, int lb) { return e >> lb; }
    __device__ static int32_t lab(T e, int lb) { return (int32_t)(e & ((1ll << lb) - 1)); }
    __device__ static T make(int64_t v, int32_t l, int lb) {
        return (v << lb) | ((int64_t)(uint32_t)l & ((1ll << lb) - 1));
    }
};
template <>
struct Elem<false> {
    using T = Pair;
    __device__ static int64_t val(const T &e, int) { return e.val; }
    __device__ static int32_t lab(const T &e, int) { return (int32_t)e.lab; }
    __device__ static T make(int64_t v, int32_t l, int) {
        T e;
        e.val = v;
        e.lab = l;
        return e;
    }
};

// One direction of the sweep for slice `slice`. FWD: t levels; else b levels.
template <int S, int T, bool FWD, bool PACKED>
__device__ void sweep_dir(const SweepArgs &a, int32_t slice, char *smem) {
    using EL = Elem<PACKED>;
    using ET = typename EL::T;
    constexpr int ACC = kSweepAccNodes;  // nodes per accumulator chunk
    constexpr int CH = kLevelWindow;     // level boundaries staged in LDS
    long long *acc = reinterpret_cast<long long *>(smem);                              // [ACC*S]
    unsigned long long *nacc = reinterpret_cast<unsigned long long *>(acc + ACC * S);  // [ACC*S]
    int32_t *slab = reinterpret_cast<int32_t *>(nacc + ACC * S);                       // [2][ACC*S]
    long long *bins = reinterpret_cast<long long *>(slab + 2 * ACC * S);               // [kBinsCap]
    LevelInfo *s_li = reinterpret_cast<LevelInfo *>(bins + kBinsCap);                  // [CH]
    __shared__ long long s_m[S];
    __shared__ int s_start[S];

    const int tid = threadIdx.x;
    const int s0 = tid % S;
    const int lb = a.lb;
    const int32_t V = a.V, L = a.L, P = a.P;
    const int64_t wbase = (int64_t)slice * V * S;
    const int32_t *lab = a.lab_w + wbase;
    ET *vals = reinterpret_cast<ET *>(FWD ? a.ftl : a.bll) + wbase;
    const int32_t *e_nb = FWD ? a.in_src : a.out_dst;
    const int32_t *e_own = FWD ? a.in_dst : a.out_src;
    const int64_t *e_cost = FWD ? a.in_cost : a.out_cost;
    const int32_t *off = FWD ? a.in_off : a.out_off;
    const bool want_nx = !FWD && a.nx_w != nullptr;
    const bool want_bins = FWD && a.K > 0;
    const bool lds_bins = want_bins && a.K * S <= kBinsCap;
    const int32_t p0 = slice * S;

    for (int i = tid; i < ACC * S; i += T) {
        acc[i] = 0;
        nacc[i] = ~0ull;
    }
    if (lds_bins)
        for (int i = tid; i < a.K * S; i += T) bins[i] = 0;

    // Records prefetched for pass 0 of a level: one edge task and one node task
    // per thread. Indices are clamped into range so the loads never branch.
    struct EdgeRec {
        int32_t nb, own, nbo;
        int64_t c;
    };
    struct NodeRec {
        int32_t ord, lab;
        int64_t comp, mem;
    };
    EdgeRec ce{0, 0, 0, 0}, ne{0, 0, 0, 0};
    NodeRec cn{0, 0, 0, 0}, nn{0, 0, 0, 0};

    auto level_at = [&](int32_t step) { return FWD ? step : L - 1 - step; };
    auto e_lo = [&](const LevelInfo &li) { return FWD ? li.in_e_lo : li.out_e_lo; };

    auto load_edge = [&](int32_t e) {
        EdgeRec r;
        r.nb = e_nb[e];
        r.own = e_own[e];
        r.c = e_cost[e];
        r.nbo = FWD ? 0 : a.out_dst_orig[e];
        return r;
    };
    auto load_node = [&](int32_t v, int s) {
        NodeRec r;
        r.ord = a.order[v];
        r.comp = a.comp_lm[v];
        r.mem = FWD ? a.mem_lm[v] : 0;
        r.lab = lab[(int64_t)v * S + s];
        return r;
    };

    // LevelInfo window [c0, c0 + CH) in LDS
    int32_t c0 = -CH;
    auto stage = [&](int32_t klo, int32_t khi) {  // make [klo, khi] resident
        if (klo >= c0 && khi < c0 + CH) return;
        __syncthreads();
        c0 = FWD ? klo : max(0, khi - CH + 1);
        for (int i = tid; i < CH; i += T)
            if (c0 + i <= L) s_li[i] = a.linfo[c0 + i];
        __syncthreads();
    };
    auto LI = [&](int32_t k) -> const LevelInfo & { return s_li[k - c0]; };

    // pass-0 loads of level k (boundaries li, ln), addresses clamped
    auto prefetch = [&](const LevelInfo &li, const LevelInfo &ln, EdgeRec &e, NodeRec &n) {
        const int32_t ea = e_lo(li), eb = e_lo(ln);
        const int32_t ei = tid < (eb - ea) * S ? ea + tid / S : (eb > ea ? ea : 0);
        const int32_t vi = tid < (ln.node_lo - li.node_lo) * S ? li.node_lo + tid / S : li.node_lo;
        e = load_edge(a.E > 0 ? ei : 0);
        n = load_node(min(vi, V - 1), s0);
    };
    // own labels of a narrow level into slab[buf]; pass 0 comes from registers
    auto fill_labels = [&](const LevelInfo &li, const LevelInfo &ln, int buf, const NodeRec &n) {
        const int32_t lo = li.node_lo, w = ln.node_lo - lo;
        int32_t *sl = slab + buf * ACC * S;
        if (tid < w * S) sl[tid] = n.lab;
        for (int32_t i = tid + T; i < w * S; i += T) sl[i] = lab[(int64_t)lo * S + i];
    };

    auto cand = [&](const ET &g, int32_t own_lab, int64_t c) {
        return EL::val(g, lb) + (EL::lab(g, lb) != own_lab ? c : 0);
    };

    auto finish_node = [&](int32_t v, int s, int32_t slot, const NodeRec &n) {
        const int64_t t = acc[slot];
        acc[slot] = 0;
        const int32_t p = p0 + s;
        if (FWD) {
            vals[(int64_t)v * S + s] = EL::make(t + n.comp, n.lab, lb);
            if (p < P) {
                if (a.direct) a.tl_out[(int64_t)n.ord * P + p] = t;
                if (want_bins) {
                    const int32_t l = n.lab;
                    if (l < 0 || l >= a.K)
                        atomicOr(a.err, 1);
                    else if (lds_bins)
                        lds_add_i64(&bins[l * S + s], n.mem);
                    else
                        atomicAdd((unsigned long long *)&a.label_mem[(int64_t)p * a.K + l],
                                  (unsigned long long)n.mem);
                }
            }
        } else {
            const int64_t b = n.comp + t;
            vals[(int64_t)v * S + s] = EL::make(b, n.lab, lb);
            if (a.direct && p < P) a.bl_out[(int64_t)n.ord * P + p] = b;
            if (want_nx) {
                const unsigned long long key = nacc[slot];
                nacc[slot] = ~0ull;
                a.nx_w[wbase + (int64_t)v * S + s] =
                    key == ~0ull ? -1 : (int32_t)(key & 0xffffffffull);
            }
        }
    };

    if (L > 0) {
        const int32_t k0 = level_at(0);
        stage(k0, k0 + 1);
        const LevelInfo li = LI(k0), ln = LI(k0 + 1);
        if (ln.node_lo - li.node_lo <= ACC) {
            prefetch(li, ln, ce, cn);
            fill_labels(li, ln, 0, cn);
        }
    }
    __syncthreads();

    for (int32_t step = 0; step < L; step++) {
        const int32_t k = level_at(step);
        const bool has_next = step + 1 < L;
        const int32_t kn = has_next ? level_at(step + 1) : k;
        stage(min(k, kn), max(k, kn) + 1);
        const int buf = step & 1;
        const LevelInfo li = LI(k), ln = LI(k + 1);
        const LevelInfo lin = LI(kn), lnn = LI(kn + 1);
        const int32_t lo = li.node_lo, hi = ln.node_lo;
        const int32_t ea = e_lo(li), eb = e_lo(ln);
        const bool next_narrow = has_next && lnn.node_lo - lin.node_lo <= ACC;

        if (hi - lo <= ACC) {
            // ---- narrow level: one chunk, pass 0 prefetched ----
            const int32_t *sl = slab + buf * ACC * S;
            const int32_t nt = (eb - ea) * S;
            const bool ev = tid < nt;
            const ET g0 = vals[ev ? (int64_t)ce.nb * S + s0 : 0];  // gather, always in range
            // issued on every path, so the wait for g0 leaves these loads in flight
            prefetch(lin, lnn, ne, nn);
            const int32_t slot0 = (ce.own - lo) * S + s0;
            int64_t c0v = 0;
            if (ev) {
                c0v = cand(g0, sl[slot0], ce.c);
                lds_max_i64(&acc[slot0], c0v);
            }
            for (int32_t i = tid + T; i < nt; i += T) {
                const EdgeRec r = load_edge(ea + i / S);
                const int s = i % S;
                const ET g = vals[(int64_t)r.nb * S + s];
                lds_max_i64(&acc[(r.own - lo) * S + s], cand(g, sl[(r.own - lo) * S + s], r.c));
            }
            __syncthreads();
            if (want_nx) {
                if (ev && c0v == acc[slot0])
                    lds_min_u64(&nacc[slot0],
                                ((unsigned long long)(uint32_t)ce.nbo << 32) | (uint32_t)ce.nb);
                for (int32_t i = tid + T; i < nt; i += T) {
                    const EdgeRec r = load_edge(ea + i / S);
                    const int s = i % S;
                    const ET g = vals[(int64_t)r.nb * S + s];
                    const int32_t slot = (r.own - lo) * S + s;
                    if (cand(g, sl[slot], r.c) == acc[slot])
                        lds_min_u64(&nacc[slot],
                                    ((unsigned long long)(uint32_t)r.nbo << 32) | (uint32_t)r.nb);
                }
                __syncthreads();
            }
            const int32_t nnt = (hi - lo) * S;
            if (tid < nnt) finish_node(lo + tid / S, s0, tid, cn);
            for (int32_t i = tid + T; i < nnt; i += T) {
                const int s = i % S;
                const int32_t v = lo + i / S;
                NodeRec r = load_node(v, s);
                r.lab = sl[i];
                finish_node(v, s, i, r);
            }
            if (next_narrow) fill_labels(lin, lnn, buf ^ 1, nn);
            __syncthreads();
        } else {
            // ---- wide level: chunks of ACC nodes, loads inline ----
            for (int32_t cn0 = lo; cn0 < hi; cn0 += ACC) {
                const int32_t cn1 = min(hi, cn0 + ACC);
                const int32_t cea = cn0 == lo ? ea : off[cn0];
                const int32_t ceb = cn1 == hi ? eb : off[cn1];
                const int32_t nt = (ceb - cea) * S;
                for (int32_t i = tid; i < nt; i += T) {
                    const EdgeRec r = load_edge(cea + i / S);
                    const int s = i % S;
                    const ET g = vals[(int64_t)r.nb * S + s];
                    lds_max_i64(&acc[(r.own - cn0) * S + s],
                                cand(g, lab[(int64_t)r.own * S + s], r.c));
                }
                __syncthreads();
                if (want_nx) {
                    for (int32_t i = tid; i < nt; i += T) {
                        const EdgeRec r = load_edge(cea + i / S);
                        const int s = i % S;
                        const ET g = vals[(int64_t)r.nb * S + s];
                        const int32_t slot = (r.own - cn0) * S + s;
                        if (cand(g, lab[(int64_t)r.own * S + s], r.c) == acc[slot])
                            lds_min_u64(&nacc[slot], ((unsigned long long)(uint32_t)r.nbo << 32) |
                                                         (uint32_t)r.nb);
                    }
                    __syncthreads();
                }
                const int32_t nnt = (cn1 - cn0) * S;
                for (int32_t i = tid; i < nnt; i += T) {
                    const int s = i % S;
                    const int32_t v = cn0 + i / S;
                    finish_node(v, s, i, load_node(v, s));
                }
                __syncthreads();
            }
            if (next_narrow) {
                prefetch(lin, lnn, ne, nn);
                fill_labels(lin, lnn, buf ^ 1, nn);
                __syncthreads();
            }
        }
        ce = ne;
        cn = nn;
    }

    if (FWD) {
        if (lds_bins) {
            __syncthreads();
            for (int i = tid; i < a.K * S; i += T) {
                const int l = i / S, s = i % S;
                if (p0 + s < P) a.label_mem[(int64_t)(p0 + s) * a.K + l] = bins[i];
            }
        }
        return;
    }
    // b direction: makespan M = max over v of tl + bl is reached at a node
    // without predecessors (tl = 0 there), i.e. at level 0; the path starts at
    // the smallest-id such node with bl == M (level 0 is sorted by id).
    if (tid < S) {
        s_m[tid] = 0;
        s_start[tid] = INT32_MAX;
    }
    __syncthreads();
    const int32_t n0 = L > 0 ? a.linfo[1].node_lo : 0;
    for (int32_t i = tid; i < n0 * S; i += T) lds_max_i64(&s_m[i % S], EL::val(vals[i], lb));
    __syncthreads();
    for (int32_t i = tid; i < n0 * S; i += T)
        if (EL::val(vals[i], lb) == s_m[i % S]) lds_min_i32(&s_start[i % S], i / S);
    __syncthreads();
    if (tid < S && p0 + tid < P) {
        a.makespan[p0 + tid] = s_m[tid];
        if (a.start) a.start[p0 + tid] = s_start[tid] == INT32_MAX ? -1 : s_start[tid];
    }
}

template <int S, int T, bool PACKED>
__global__ __launch_bounds__(T) void k_sweep(SweepArgs a) {
    extern __shared__ __align__(16) char smem[];
    const int32_t n_slices = (a.P + S - 1) / S;
    if ((int32_t)blockIdx.x < n_slices)
        sweep_dir<S, T, false, PACKED>(a, blockIdx.x, smem);
    else
        sweep_dir<S, T, true, PACKED>(a, blockIdx.x - n_slices, smem);
}

template <int S>
constexpr size_t sweep_lds_bytes() {
    return (size_t)kSweepAccNodes * S * 8 * 2 + (size_t)kSweepAccNodes * S * 4 * 2 +
           (size_t)kBinsCap * 8 + (size_t)kLevelWindow * sizeof(LevelInfo);
}

// Outputs in the caller's layout: tl, bl [V][P] in original ids and the
// critical flags crit = (tl + bl == M_p). A 32-node x 64-placement tile goes
// through LDS so that the slice-major workspace is read contiguously and each
// output row order[v] is written as one contiguous 512-byte run.
template <int S, bool PACKED>
__global__ __launch_bounds__(256) void k_emit(SweepArgs a, uint8_t *crit) {
    using EL = Elem<PACKED>;
    using ET = typename EL::T;
    constexpr int TV = 32, TP = 64;
    __shared__ long long t_tl[TV][TP + 1];
    __shared__ long long t_bl[TV][TP + 1];
    const int32_t V = a.V, P = a.P;
    const int32_t v0 = blockIdx.x * TV, q0 = blockIdx.y * TP;
    const int32_t sl0 = q0 / S;
    const int n_sl = min(TP / S, (P + S - 1) / S - sl0);
    const ET *ft = reinterpret_cast<const ET *>(a.ftl);
    const ET *bl = reinterpret_cast<const ET *>(a.bll);
    for (int i = threadIdx.x; i < n_sl * TV * S; i += 256) {
        const int sl = i / (TV * S), j = i % (TV * S);
        const int r = j / S, s = j % S;
        const int32_t v = v0 + r;
        if (v < V) {
            const int64_t idx = ((int64_t)(sl0 + sl) * V + v) * S + s;
            t_tl[r][sl * S + s] = EL::val(ft[idx], a.lb) - a.comp_lm[v];
            t_bl[r][sl * S + s] = EL::val(bl[idx], a.lb);
        }
    }
    __syncthreads();
    for (int i = threadIdx.x; i < TV * TP; i += 256) {
        const int r = i / TP, q = i % TP;
        const int32_t v = v0 + r, p = q0 + q;
        if (v < V && p < P) {
            const int64_t o = (int64_t)a.order[v] * P + p;
            const int64_t t = t_tl[r][q], b = t_bl[r][q];
            a.tl_out[o] = t;
            a.bl_out[o] = b;
            if (crit) crit[o] = (uint8_t)(t + b == a.makespan[p]);
        }
    }
}

// One wave per placement walks the chosen-successor links from the path
// start. Links point to strictly later levels (larger level-major ids), so the
// wave stages a window of its links in LDS with coalesced loads, lane 0
// chases inside the window, and the window moves forward when the walk leaves
// it.
template <int S>
__global__ __launch_bounds__(256) void k_chase_batch(int32_t V, int32_t P, const int32_t *order,
                                                     const int32_t *nx_w, const int32_t *start,
                                                     int32_t *path, int32_t stride,
                                                     int32_t *path_len) {
    constexpr int kWin = 2048;
    __shared__ int32_t win[256 / kWave][kWin];
    const int lane = lane_id(), w = wave_id();
    const int32_t p = blockIdx.x * (256 / kWave) + w;
    if (p >= P) return;
    const int32_t slice = p / S, s = p % S;
    const int32_t *nx = nx_w + (int64_t)slice * V * S;
    int32_t *out = path + (int64_t)p * stride;
    int32_t cur = start[p], len = 0, mine = -1;
    // The walk is uniform across the wave; lane i keeps the (i mod 64)-th path
    // node and the wave writes 64 original ids at a time.
    while (cur >= 0) {
        const int32_t base = cur;
        for (int i = lane; i < kWin; i += kWave)
            win[w][i] = base + i < V ? nx[(int64_t)(base + i) * S + s] : -1;
        __builtin_amdgcn_wave_barrier();
        int32_t c = base;
        while (c >= base && c < base + kWin) {
            if ((len & (kWave - 1)) == lane) mine = c;
            len++;
            if ((len & (kWave - 1)) == 0) out[len - kWave + lane] = order[mine];
            const int32_t n = win[w][c - base];
            c = n > c ? n : -1;  // links go to strictly later levels
        }
        cur = c;
        __builtin_amdgcn_wave_barrier();
    }
    const int32_t r = len & (kWave - 1);
    if (lane < r) out[len - r + lane] = order[mine];
    if (lane == 0) path_len[p] = len;
}

constexpr int kSingleThreads = 512;
constexpr int kBatchSlots = 2;
constexpr int kBatchThreads = 256;

}  // namespace

hipError_t launch_permute_labels(const Graph &g, const int32_t *placement, int32_t *lab_lm) {
    return launch_permute_labels_batch(g, placement, 1, 1, lab_lm);
}

hipError_t launch_permute_labels_batch(const Graph &g, const int32_t *placements, int32_t P,
                                       int32_t S, int32_t *lab_w) {
    if (g.V == 0 || P == 0) return hipSuccess;
    dim3 grid((g.V + 63) / 64, (P + 63) / 64);
    if (S == 1)
        k_permute_labels<1><<<grid, 256, 0, g.stream>>>(g.V, P, g.order, placements, lab_w);
    else if (S == kBatchSlots)
        k_permute_labels<kBatchSlots><<<grid, 256, 0, g.stream>>>(g.V, P, g.order, placements,
                                                                  lab_w);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

int batch_slots() { return kBatchSlots; }

hipError_t launch_sweep(const SweepArgs &a, int32_t S, hipStream_t s) {
    const int32_t n_slices = (a.P + S - 1) / S;
    if (n_slices == 0) return hipSuccess;
    const bool packed = a.lb > 0;
    if (S == 1 && !packed) {
        k_sweep<1, kSingleThreads, false>
            <<<2 * n_slices, kSingleThreads, sweep_lds_bytes<1>(), s>>>(a);
    } else if (S == kBatchSlots && packed) {
        k_sweep<kBatchSlots, kBatchThreads, true>
            <<<2 * n_slices, kBatchThreads, sweep_lds_bytes<kBatchSlots>(), s>>>(a);
    } else if (S == kBatchSlots && !packed) {
        k_sweep<kBatchSlots, kBatchThreads, false>
            <<<2 * n_slices, kBatchThreads, sweep_lds_bytes<kBatchSlots>(), s>>>(a);
    } else {
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_emit(const SweepArgs &a, int32_t S, uint8_t *crit, hipStream_t s) {
    if ((int64_t)a.V * a.P == 0) return hipSuccess;
    if (S != kBatchSlots) return hipErrorInvalidValue;
    dim3 grid((a.V + 31) / 32, (a.P + 63) / 64);
    if (a.lb > 0)
        k_emit<kBatchSlots, true><<<grid, 256, 0, s>>>(a, crit);
    else
        k_emit<kBatchSlots, false><<<grid, 256, 0, s>>>(a, crit);
    return hipGetLastError();
}

hipError_t launch_chase_batch(const SweepArgs &a, int32_t S, const int32_t *order, int32_t *path,
                              int32_t stride, int32_t *path_len, hipStream_t s) {
    if (a.P == 0) return hipSuccess;
    const int per_block = 256 / kWave;
    const unsigned grid = (unsigned)((a.P + per_block - 1) / per_block);
    if (S == 1)
        k_chase_batch<1><<<grid, 256, 0, s>>>(a.V, a.P, order, a.nx_w, a.start, path, stride,
                                              path_len);
    else if (S == kBatchSlots)
        k_chase_batch<kBatchSlots><<<grid, 256, 0, s>>>(a.V, a.P, order, a.nx_w, a.start, path,
                                                        stride, path_len);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

}  // namespace pardnn
