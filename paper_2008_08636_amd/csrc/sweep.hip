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
#include "sweep_common.h"

#include <type_traits>

namespace pardnn {

namespace {

constexpr int kChaseRegs = 16;   // registers per lane of a path-walk window
constexpr int kEmitNodes = 32;   // level-major nodes per emit workgroup
constexpr int kEmitCols = 128;   // placements per emit chunk

// Lanes of one placement slice: labels gathered into the slice-major layout
// [slice][V][S] through an LDS tile, so that both the reads of the caller's
// placement rows and the writes are contiguous.
template <int S>
__global__ __launch_bounds__(256) void k_permute_labels(int32_t V, int32_t P,
                                                        const int32_t *order,
                                                        const int32_t *placements,
                                                        int32_t *lab_w, int64_t lab_stride,
                                                        int32_t K, int32_t *err, int32_t *fit,
                                                        uint32_t fit_limit, int lab16,
                                                        const int32_t *gate, int32_t gate_want) {
    if (gate != nullptr && *gate != gate_want) return;   // (uniform)
    constexpr int TV = 64, TP = 64;  // tile: 64 nodes x 64 placements
    __shared__ int32_t tile[TV][TP + 1];
    const int32_t n_slices = (P + S - 1) / S;
    const int32_t v0 = blockIdx.x * TV;
    const int32_t q0 = blockIdx.y * TP;  // first placement of the tile
    const int tx = threadIdx.x & (TP - 1), ty = threadIdx.x / TP;
    for (int r = ty; r < TV; r += 256 / TP) {
        const int32_t v = v0 + r, p = q0 + tx;
        int32_t x = 0;
        if (v < V && p < P) {
            x = placements[(int64_t)order[v] * P + p];
            if (K > 0 && (x < 0 || x >= K)) atomicOr(err, 1);
            if (fit != nullptr && (uint32_t)x >= fit_limit) *fit = 0;
        }
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
        const int64_t o = (int64_t)(sl0 + sl) * lab_stride + (int64_t)v * S + s;
        if (v >= V) continue;
        // streamed past L2, as the sweep reads it much later; 16-bit labels
        // were checked against their full values above
        if (lab16)
            __builtin_nontemporal_store((uint16_t)tile[r][sl * S + s],
                                        reinterpret_cast<uint16_t *>(lab_w) + o);
        else
            __builtin_nontemporal_store(tile[r][sl * S + s], &lab_w[o]);
    }
}

// LDS bytes of one sweep workgroup.
template <int S, int ACC, bool PACKED>
constexpr size_t sweep_lds_bytes() {
    using ET = typename Elem<PACKED>::T;
    return (size_t)2 * ACC * S * 8          // acc (double-buffered by step parity)
           + (size_t)ACC * S * 8            // nacc
           + (size_t)2 * ACC * S * 4        // slab
           + (size_t)2 * ACC * S * sizeof(ET)  // nbuf
           + (size_t)kBinsCap * 8 + (size_t)kLevelWindow * sizeof(LevelInfo);
}

// One direction of the sweep for slice `slice`. FWD: t levels; else b levels.
//
// Per narrow level k (at most ACC nodes) a step is:
//   edge phase: every (edge, slot) task folds its candidate into acc[k & 1]
//     with an LDS max. The neighbour value comes from nbuf (LDS) when the
//     neighbour lies on the level computed in the previous step, or from a
//     register loaded one step earlier when it lies further back. So no global
//     load sits on the critical path of a narrow level.
//   barrier
//   node phase: each (node, slot) reads its accumulator, writes its value to
//     the workspace (global) and to nbuf (for the next level), and clears the
//     accumulators of the previous level.
//   barrier
// While a step runs, the records of level k+2 and the far neighbour values
// of level k+1 are loaded into registers. Two edge tasks per thread are
// pipelined this way; further ones (levels with more than 2T tasks) load
// inline. Levels wider than ACC nodes go through a chunked path without
// pipelining.
//
// The b direction must also pick, among the successors reaching the max, the
// one with the smallest original id (the next node of the critical path).
// PACKED folds that into the max itself: key = (value << ob) | (omax - orig),
// and the node phase reads the successor's original id back from the low
// bits of the maximum. Otherwise a second LDS phase takes the min over the
// tied successors.
template <int S, int T, int ACC, bool FWD, bool PACKED>
__device__ void sweep_dir(const SweepArgs &a, int32_t slice, char *smem) {
    constexpr bool DIRECT = S == 1;  // one placement: write tl/bl straight to the caller
    using EL = Elem<PACKED>;
    using ET = typename EL::T;
    constexpr int CH = kLevelWindow;
    long long *acc = reinterpret_cast<long long *>(smem);                                  // [2][ACC*S]
    unsigned long long *nacc = reinterpret_cast<unsigned long long *>(acc + 2 * ACC * S);  // [ACC*S]
    int32_t *slab = reinterpret_cast<int32_t *>(nacc + ACC * S);                           // [2][ACC*S]
    ET *nbuf = reinterpret_cast<ET *>(slab + 2 * ACC * S);                                 // [2][ACC*S]
    long long *bins = reinterpret_cast<long long *>(nbuf + 2 * ACC * S);                   // [kBinsCap]
    LevelInfo *s_li = reinterpret_cast<LevelInfo *>(bins + kBinsCap);                      // [CH]
    __shared__ long long s_m[S];
    __shared__ int s_start[S];

    const int tid = threadIdx.x;
    const int s0 = tid % S;
    const int lb = a.lb;
    const int ob = PACKED && !FWD ? a.ob : 0;
    const long long omax = (1ll << ob) - 1;
    const int32_t V = a.V, L = a.L, P = a.P;
    const int64_t wbase = (int64_t)slice * a.ws_stride;
    const int32_t *lab = a.lab_w + (int64_t)slice * a.lab_stride;
    ET *vals = reinterpret_cast<ET *>(FWD ? a.ftl : a.bll) + wbase;
    const EdgeRec16 *erec = FWD ? a.in_rec : a.out_rec;
    const int32_t *off = FWD ? a.in_off : a.out_off;
    const bool want_nx = !FWD && a.nx_w != nullptr;
    int32_t *nxb = want_nx ? a.nx_w + wbase : nullptr;
    const bool tie_phase = want_nx && !PACKED;
    const bool want_bins = FWD && a.K > 0;
    const bool lds_bins = want_bins && a.K * S <= kBinsCap;
    const int32_t p0 = slice * S;

    for (int i = tid; i < 2 * ACC * S; i += T) acc[i] = 0;
    for (int i = tid; i < ACC * S; i += T) nacc[i] = ~0ull;
    if (lds_bins)
        for (int i = tid; i < a.K * S; i += T) bins[i] = 0;

    struct EdgeRec {
        int32_t nb, own, nbo;
        int64_t c;
    };
    struct NodeRec {
        int32_t ord, lab;
        int64_t comp, mem;
    };
    struct Recs {        // prefetched records of one level: two edge tasks, one node task
        EdgeRec e0, e1;
        NodeRec n;
    };

    auto level_at = [&](int32_t step) { return FWD ? step : L - 1 - step; };
    auto e_lo = [&](const LevelInfo &li) { return FWD ? li.in_e_lo : li.out_e_lo; };

    // one 16-byte load per edge record (plus the successor's id for b)
    auto load_edge = [&](int32_t e) {
        const EdgeRec16 x = at(erec, (uint32_t)e);
        EdgeRec r;
        r.nb = x.nb;
        r.own = x.own;
        r.c = x.cost;
        r.nbo = FWD ? 0 : at(a.out_dst_orig, (uint32_t)e);
        return r;
    };
    // one 16-byte load of the node constants, the label, and (single
    // placement only) the node's original id for the direct outputs
    auto load_node = [&](int32_t v, int s) {
        const NodeRec16 x = at(a.node_rec, (uint32_t)v);
        NodeRec r;
        r.ord = DIRECT ? at(a.order, (uint32_t)v) : 0;
        r.comp = x.comp;
        r.mem = x.mem;
        r.lab = at(lab, (uint32_t)(v * S + s));
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
    auto LI = [&](int32_t k) -> LevelInfo { return s_li[k - c0]; };

    // records of a level (boundaries li, ln), addresses clamped into range
    auto prefetch = [&](const LevelInfo &li, const LevelInfo &ln, Recs &r) {
        const int32_t ea = e_lo(li), eb = e_lo(ln);
        const int32_t nt = (eb - ea) * S;
        const int32_t e0 = tid < nt ? ea + tid / S : 0;
        const int32_t e1 = tid + T < nt ? ea + (tid + T) / S : 0;
        const int32_t vi = tid < (ln.node_lo - li.node_lo) * S ? li.node_lo + tid / S : 0;
        r.e0 = load_edge(a.E > 0 ? e0 : 0);
        r.e1 = load_edge(a.E > 0 ? e1 : 0);
        r.n = load_node(min(vi, V - 1), s0);
    };
    auto fill_labels = [&](const LevelInfo &li, const LevelInfo &ln, int buf, const NodeRec &n) {
        const int32_t lo = li.node_lo, w = ln.node_lo - lo;
        int32_t *sl = slab + buf * ACC * S;
        if (tid < w * S) sl[tid] = n.lab;
        for (int32_t i = tid + T; i < w * S; i += T) sl[i] = at(lab, (uint32_t)(lo * S + i));
    };
    auto cand = [&](const ET &g, int32_t own_lab, int64_t c) {
        return EL::val(g, lb) + (EL::lab(g, lb) != own_lab ? c : 0);
    };
    // accumulator key of a candidate (b, PACKED: with the successor's id)
    auto akey = [&](int64_t cv, int32_t nbo) -> long long {
        return PACKED && !FWD ? (cv << ob) | (omax - nbo) : cv;
    };
    auto akey_val = [&](long long key) -> int64_t { return PACKED && !FWD ? key >> ob : key; };

    auto finish_node = [&](int32_t v, int s, int32_t slot, long long key, const NodeRec &n,
                           ET *nb_out) {
        const int64_t t = akey_val(key);
        const int32_t p = p0 + s;
        if (FWD) {
            const ET out = EL::make(t + n.comp, n.lab, lb);
            at(vals, (uint32_t)(v * S + s)) = out;
            if (nb_out) nb_out[slot] = out;
            if (p < P) {
                if (DIRECT) a.tl_out[(int64_t)n.ord * P + p] = t;
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
            const ET out = EL::make(b, n.lab, lb);
            at(vals, (uint32_t)(v * S + s)) = out;
            if (nb_out) nb_out[slot] = out;
            if (DIRECT && p < P) a.bl_out[(int64_t)n.ord * P + p] = b;
            // successor on the canonical path, as an original id: PACKED keys
            // carry it in their low bits, else the tie phase left it in nacc
            if (want_nx) {
                if (PACKED) {
                    at(nxb, (uint32_t)(v * S + s)) = key == 0 ? -1 : (int32_t)(omax - (key & omax));
                } else {
                    const unsigned long long k2 = nacc[slot];
                    nacc[slot] = ~0ull;
                    at(nxb, (uint32_t)(v * S + s)) = k2 == ~0ull ? -1 : (int32_t)(k2 >> 32);
                }
            }
        }
    };

    // ---- pipeline state ----
    // One set per level in flight: level k (consumed now), k+1 (its far values
    // are being loaded) and k+2 (its records are being loaded). The step loop
    // is unrolled three times and the sets rotate by name, so no register that
    // a load is still filling is ever copied: such a copy would make the wave
    // wait for every load in flight and drain the pipeline at each level.
    struct Stage {
        Recs r;            // records of the level, loaded two steps ahead
        ET f0, f1;         // far neighbour values of the two pipelined tasks
        bool h0, h1;       // the task's neighbour is far (value in f0 / f1)
        LevelInfo li, ln;  // the level's boundaries and the next level's
    };
    Stage SA{}, SB{}, SC{};
    if (L > 0) {
        const int32_t k0 = level_at(0), k1 = L > 1 ? level_at(1) : k0;
        stage(min(k0, k1), max(k0, k1) + 1);
        SA.li = LI(k0);
        SA.ln = LI(k0 + 1);
        SB.li = LI(k1);
        SB.ln = LI(k1 + 1);
        prefetch(SA.li, SA.ln, SA.r);
        prefetch(SB.li, SB.ln, SB.r);
        if (SA.ln.node_lo - SA.li.node_lo <= ACC) fill_labels(SA.li, SA.ln, 0, SA.r.n);
    }
    __syncthreads();
    int32_t plo = 0, phi = 0;     // previous level's node range
    bool prev_in_lds = false;     // previous level's values sit in nbuf[(step - 1) & 1]

    auto body = [&](int32_t step, Stage &A, Stage &B, Stage &C) __attribute__((always_inline)) {
        const bool has_next = step + 1 < L;
        const int32_t k = level_at(step);
        const int32_t knn = step + 2 < L ? level_at(step + 2) : (has_next ? level_at(step + 1) : k);
        stage(min(k, knn), max(k, knn) + 1);
        C.li = LI(knn);
        C.ln = LI(knn + 1);
        const int buf = step & 1;
        const int32_t lo = A.li.node_lo, hi = A.ln.node_lo;
        const int32_t ea = e_lo(A.li), eb = e_lo(A.ln);
        const int32_t nt = (eb - ea) * S;
        const int32_t nt_next = (e_lo(B.ln) - e_lo(B.li)) * S;
        const bool next_narrow = has_next && B.ln.node_lo - B.li.node_lo <= ACC;
        long long *accb = acc + buf * ACC * S;
        long long *accp = acc + (buf ^ 1) * ACC * S;
        const ET *nprev = nbuf + (buf ^ 1) * ACC * S;
        const int sB = (tid + T) % S;

        // neighbour value of an inline task: near in LDS, else global
        auto nval = [&](const EdgeRec &r, int s) -> ET {
            if (prev_in_lds && r.nb >= plo && r.nb < phi) return nprev[(r.nb - plo) * S + s];
            return at(vals, (uint32_t)(r.nb * S + s));
        };

        if (__builtin_expect(hi - lo <= ACC, 1)) {
            // ---- narrow level ----
            const int32_t *sl = slab + buf * ACC * S;
            const bool ev0 = tid < nt, ev1 = tid + T < nt;
            long long k0v = 0, k1v = 0;
            // pass 0/1 neighbours: prefetched register (far, or everything after a
            // wide level) or the previous level's values in LDS -- no global load
            const ET l0 = nprev[ev0 && !A.h0 ? (A.r.e0.nb - plo) * S + s0 : 0];
            const ET l1 = nprev[ev1 && !A.h1 ? (A.r.e1.nb - plo) * S + sB : 0];
            if (ev0) {
                const ET g = A.h0 ? A.f0 : l0;
                k0v = akey(cand(g, sl[(A.r.e0.own - lo) * S + s0], A.r.e0.c), A.r.e0.nbo);
                lds_max_i64(&accb[(A.r.e0.own - lo) * S + s0], k0v);
            }
            if (ev1) {
                const ET g = A.h1 ? A.f1 : l1;
                k1v = akey(cand(g, sl[(A.r.e1.own - lo) * S + sB], A.r.e1.c), A.r.e1.nbo);
                lds_max_i64(&accb[(A.r.e1.own - lo) * S + sB], k1v);
            }
            // next level's far neighbours (final already) and level k+2's records
            B.h0 = has_next && tid < nt_next && (FWD ? B.r.e0.nb < lo : B.r.e0.nb >= hi);
            B.h1 = has_next && tid + T < nt_next && (FWD ? B.r.e1.nb < lo : B.r.e1.nb >= hi);
            B.f0 = at(vals, B.h0 ? (uint32_t)(B.r.e0.nb * S + s0) : 0u);
            B.f1 = at(vals, B.h1 ? (uint32_t)(B.r.e1.nb * S + sB) : 0u);
            prefetch(C.li, C.ln, C.r);
            for (int32_t i = tid + 2 * T; i < nt; i += T) {
                const EdgeRec r = load_edge(ea + i / S);
                const int s = i % S;
                const ET g = nval(r, s);
                lds_max_i64(&accb[(r.own - lo) * S + s],
                            akey(cand(g, sl[(r.own - lo) * S + s], r.c), r.nbo));
            }
            __syncthreads();
            if (tie_phase) {
                if (ev0 && k0v == accb[(A.r.e0.own - lo) * S + s0])
                    lds_min_u64(&nacc[(A.r.e0.own - lo) * S + s0],
                                ((unsigned long long)(uint32_t)A.r.e0.nbo << 32) | (uint32_t)A.r.e0.nb);
                if (ev1 && k1v == accb[(A.r.e1.own - lo) * S + sB])
                    lds_min_u64(&nacc[(A.r.e1.own - lo) * S + sB],
                                ((unsigned long long)(uint32_t)A.r.e1.nbo << 32) | (uint32_t)A.r.e1.nb);
                for (int32_t i = tid + 2 * T; i < nt; i += T) {
                    const EdgeRec r = load_edge(ea + i / S);
                    const int s = i % S;
                    const ET g = nval(r, s);
                    const int32_t slot = (r.own - lo) * S + s;
                    if (akey(cand(g, sl[slot], r.c), r.nbo) == accb[slot])
                        lds_min_u64(&nacc[slot],
                                    ((unsigned long long)(uint32_t)r.nbo << 32) | (uint32_t)r.nb);
                }
                __syncthreads();
            }
            ET *nb_out = nbuf + buf * ACC * S;
            const int32_t nnt = (hi - lo) * S;
            if (tid < nnt) finish_node(lo + tid / S, s0, tid, accb[tid], A.r.n, nb_out);
            for (int32_t i = tid + T; i < nnt; i += T) {
                const int s = i % S;
                const int32_t v = lo + i / S;
                NodeRec r = load_node(v, s);
                r.lab = sl[i];
                finish_node(v, s, i, accb[i], r, nb_out);
            }
            // clear the previous level's accumulators (used again at step + 1)
            for (int32_t i = tid; i < (phi - plo) * S && phi - plo <= ACC; i += T) accp[i] = 0;
            if (next_narrow) fill_labels(B.li, B.ln, buf ^ 1, B.r.n);
            __syncthreads();
            prev_in_lds = true;
        } else {
            // ---- wide level: chunks of ACC nodes, loads inline ----
            if (phi - plo <= ACC)
                for (int32_t i = tid; i < (phi - plo) * S; i += T) accp[i] = 0;
            __syncthreads();
            for (int32_t cn0 = lo; cn0 < hi; cn0 += ACC) {
                const int32_t cn1 = min(hi, cn0 + ACC);
                const int32_t cea = cn0 == lo ? ea : off[cn0];
                const int32_t ceb = cn1 == hi ? eb : off[cn1];
                const int32_t cnt = (ceb - cea) * S;
                for (int32_t i = tid; i < cnt; i += T) {
                    const EdgeRec r = load_edge(cea + i / S);
                    const int s = i % S;
                    const ET g = nval(r, s);
                    lds_max_i64(&accb[(r.own - cn0) * S + s],
                                akey(cand(g, at(lab, (uint32_t)(r.own * S + s)), r.c), r.nbo));
                }
                __syncthreads();
                if (tie_phase) {
                    for (int32_t i = tid; i < cnt; i += T) {
                        const EdgeRec r = load_edge(cea + i / S);
                        const int s = i % S;
                        const ET g = nval(r, s);
                        const int32_t slot = (r.own - cn0) * S + s;
                        if (akey(cand(g, at(lab, (uint32_t)(r.own * S + s)), r.c), r.nbo) == accb[slot])
                            lds_min_u64(&nacc[slot],
                                        ((unsigned long long)(uint32_t)r.nbo << 32) | (uint32_t)r.nb);
                    }
                    __syncthreads();
                }
                const int32_t cnn = (cn1 - cn0) * S;
                for (int32_t i = tid; i < cnn; i += T) {
                    const int s = i % S;
                    const int32_t v = cn0 + i / S;
                    finish_node(v, s, i, accb[i], load_node(v, s), nullptr);
                }
                __syncthreads();
                for (int32_t i = tid; i < cnn; i += T) accb[i] = 0;
                __syncthreads();
            }
            // the wide level is final now: fetch every neighbour of the next
            // level's pipelined tasks, near ones included
            B.h0 = has_next && tid < nt_next;
            B.h1 = has_next && tid + T < nt_next;
            B.f0 = at(vals, B.h0 ? (uint32_t)(B.r.e0.nb * S + s0) : 0u);
            B.f1 = at(vals, B.h1 ? (uint32_t)(B.r.e1.nb * S + sB) : 0u);
            prefetch(C.li, C.ln, C.r);
            if (next_narrow) fill_labels(B.li, B.ln, buf ^ 1, B.r.n);
            __syncthreads();
            prev_in_lds = false;
        }
        plo = lo;
        phi = hi;
    };
    int32_t step = 0;
    for (; step + 3 <= L; step += 3) {
        body(step, SA, SB, SC);
        body(step + 1, SB, SC, SA);
        body(step + 2, SC, SA, SB);
    }
    for (; step < L; step++) {  // the last L mod 3 levels: rotate by copying
        body(step, SA, SB, SC);
        const Stage t = SA;
        SA = SB;
        SB = SC;
        SC = t;
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

template <int S, int T, int ACC, bool PACKED>
__global__ __launch_bounds__(T) void k_sweep(SweepArgs a) {
    extern __shared__ __align__(16) char smem[];
    if (a.gate != nullptr && *a.gate != a.gate_want) return;
    const int32_t n_slices = (a.P + S - 1) / S;
    if ((int32_t)blockIdx.x < n_slices)
        sweep_dir<S, T, ACC, false, PACKED>(a, blockIdx.x, smem);
    else
        sweep_dir<S, T, ACC, true, PACKED>(a, blockIdx.x - n_slices, smem);
}

// Outputs in the caller's layout: tl, bl [V][P] in original ids and the
// critical flags crit = (tl + bl == M_p). A workgroup owns TV level-major
// nodes and walks the placements in chunks of TP: a chunk goes through an LDS
// tile so that the slice-major workspace is read contiguously and each output
// row order[v] is written as one contiguous run. All of a row is written by
// one workgroup, in order, so the partial lines of neighbouring chunks (the
// byte-wide flags) meet in the same L2. The loads of the next chunk are in
// flight while the current one is stored. When `cbits` is given, the flags of
// the workgroup's nodes also go out as TV / 32 bit words per placement,
// cbits[p][w] (bit r of word w: level-major node 32 w + r), for the path
// walk; node groups are assigned so that the workgroups of one XCD (every 8th
// workgroup) take consecutive groups, so that the words of one placement row
// meet in that XCD's L2.
template <int TV, int TP>
constexpr int emit_lds() {
    return 2 * TV * (TP + 1) * 8 + TV * 4 + TV * 8 + TP * 8;
}

template <int S, bool PACKED, int TV, int TP>
__device__ void emit_rows(const SweepArgs &a, uint8_t *crit, uint32_t *cbits, int32_t bx,
                          char *smem) {
    using EL = Elem<PACKED>;
    using ET = typename EL::T;
    using BW = typename std::conditional<TV == 64, unsigned long long, uint32_t>::type;
    constexpr int NT = 256;
    constexpr int PER = TV * TP / NT;  // elements per thread and chunk
    static_assert(NT % TP == 0, "a thread keeps one placement column");
    static_assert(TV == 32 || TV == 64, "one or two bit words per placement");
    long long(*t_tl)[TP + 1] = reinterpret_cast<long long(*)[TP + 1]>(smem);
    long long(*t_bl)[TP + 1] = reinterpret_cast<long long(*)[TP + 1]>(smem + TV * (TP + 1) * 8);
    int32_t *s_ord = reinterpret_cast<int32_t *>(smem + 2 * TV * (TP + 1) * 8);
    long long *s_comp = reinterpret_cast<long long *>(s_ord + TV);
    BW *s_bits = reinterpret_cast<BW *>(s_comp + TV);   // [TP]
    const int tid = threadIdx.x, col = tid % TP;
    const int32_t V = a.V, P = a.P;
    const int32_t v0 = bx * TV;
    const int32_t n_words = (V + 31) / 32;
    const int32_t n_slices = (P + S - 1) / S;
    const int32_t n_chunks = (P + TP - 1) / TP;
    const ET *ft = reinterpret_cast<const ET *>(a.ftl);
    const ET *bl = reinterpret_cast<const ET *>(a.bll);
    const int bfo = PACKED && a.nxf ? a.ob : 0;   // successor links below the label bits
    if (tid < TV) {
        const int32_t v = min(v0 + tid, V - 1);
        s_ord[tid] = a.order[v];
        s_comp[tid] = a.comp_lm[v];
    }
    if (tid < TP) s_bits[tid] = 0;
    // element i of a chunk read: slice i / (TV S), node (i % (TV S)) / S, slot i % S
    ET fv[PER], bv[PER];
    auto load = [&](int32_t ch) {
        const int32_t sl0 = ch * (TP / S);
#pragma unroll
        for (int j = 0; j < PER; j++) {
            const int i = tid + j * NT;
            const int sl = i / (TV * S), r = (i % (TV * S)) / S, s2 = i % S;
            const int64_t idx = (int64_t)min(sl0 + sl, n_slices - 1) * a.ws_stride +
                                (int64_t)min(v0 + r, V - 1) * S + s2;
            if constexpr (PACKED) {   // read once: no need to keep the lines
                fv[j] = __builtin_nontemporal_load(&ft[idx]);
                bv[j] = __builtin_nontemporal_load(&bl[idx]);
            } else {
                fv[j] = ft[idx];
                bv[j] = bl[idx];
            }
        }
    };
    load(0);
    for (int32_t ch = 0; ch < n_chunks; ch++) {
        __syncthreads();   // the tiles are free (and s_ord, s_comp, s_bits are set)
#pragma unroll
        for (int j = 0; j < PER; j++) {
            const int i = tid + j * NT;
            const int sl = i / (TV * S), r = (i % (TV * S)) / S, s2 = i % S;
            t_tl[r][sl * S + s2] = EL::val(fv[j], a.lb) - s_comp[r];
            t_bl[r][sl * S + s2] = EL::val(bv[j], a.lb) >> bfo;
        }
        if (ch + 1 < n_chunks) load(ch + 1);
        const int32_t p = ch * TP + col;   // this thread's placement column
        const int64_t m = a.makespan[min(p, P - 1)];
        __syncthreads();
        BW bits = 0;
        if (p < P) {
#pragma unroll
            for (int j = 0; j < PER; j++) {
                const int r = (tid + j * NT) / TP;
                if (v0 + r < V) {
                    const int64_t o = (int64_t)s_ord[r] * P + p;
                    const int64_t t = t_tl[r][col], b = t_bl[r][col];
                    // optional outputs, written once and streamed past the
                    // caches; the byte flags stay ordinary stores so that
                    // their partial lines merge in L2
                    if (a.tl_out) __builtin_nontemporal_store(t, &a.tl_out[o]);
                    if (a.bl_out) __builtin_nontemporal_store(b, &a.bl_out[o]);
                    const bool c = t + b == m;
                    if (crit) crit[o] = (uint8_t)c;
                    bits |= (BW)c << r;
                }
            }
        }
        if (cbits != nullptr) {
            __hip_atomic_fetch_or(&s_bits[col], bits, __ATOMIC_RELAXED,
                                  __HIP_MEMORY_SCOPE_WORKGROUP);
            __syncthreads();
            if (tid < TP) {
                if (p < P) {
                    const BW x = s_bits[tid];
                    uint32_t *row = cbits + (int64_t)p * n_words + bx * (TV / 32);
                    row[0] = (uint32_t)x;
                    if (TV == 64 && bx * 2 + 1 < n_words) row[1] = (uint32_t)((uint64_t)x >> 32);
                }
                s_bits[tid] = 0;
            }
        }
    }
}

// The same outputs for the batched pair sweep (two slots per slice, packed
// values), 16 bytes per lane: a thread reads both slots of one node of a
// slice, and writes two adjacent placements of one output row (and their two
// flag bytes), so that every request carries twice the bytes of the general
// version. With an odd number of placements the rows are not 16-byte
// aligned, and the stores fall back to 8-byte (and single-byte) ones.
template <int TV, int TP>
__device__ void emit_rows_pair(const SweepArgs &a, uint8_t *crit, uint32_t *cbits, int32_t bx,
                               char *smem) {
    using EL = Elem<true>;
    using BW = typename std::conditional<TV == 64, unsigned long long, uint32_t>::type;
    typedef long long v2i64 __attribute__((ext_vector_type(2)));
    constexpr int S = 2, NT = 256, NW = NT / kWave;
    constexpr int PER = TV * TP / S / NT;   // 16-byte loads per thread and array
    constexpr int RPW = TV / NW;            // output rows per wave
    static_assert(TP == 2 * kWave, "a lane writes two placements of a row");
    static_assert(TV == 32 || TV == 64, "one or two bit words per placement");
    long long(*t_tl)[TP + 1] = reinterpret_cast<long long(*)[TP + 1]>(smem);
    long long(*t_bl)[TP + 1] = reinterpret_cast<long long(*)[TP + 1]>(smem + TV * (TP + 1) * 8);
    int32_t *s_ord = reinterpret_cast<int32_t *>(smem + 2 * TV * (TP + 1) * 8);
    long long *s_comp = reinterpret_cast<long long *>(s_ord + TV);
    BW *s_bits = reinterpret_cast<BW *>(s_comp + TV);   // [TP]
    const int tid = threadIdx.x, lane = lane_id(), w = wave_id();
    const int32_t V = a.V, P = a.P;
    const int32_t v0 = bx * TV;
    const int32_t n_words = (V + 31) / 32;
    const int32_t n_slices = (P + S - 1) / S;
    const int32_t n_chunks = (P + TP - 1) / TP;
    const bool even = (P & 1) == 0;
    const int bfo = a.nxf ? a.ob : 0;   // successor links below the label bits
    if (tid < TV) {
        const int32_t v = min(v0 + tid, V - 1);
        s_ord[tid] = a.order[v];
        s_comp[tid] = a.comp_lm[v];
    }
    if (tid < TP) s_bits[tid] = 0;
    // load j of a chunk: slice (tid + j NT) / TV, node (tid + j NT) % TV
    v2i64 fv[PER], bv[PER];
    auto load = [&](int32_t ch) {
        const int32_t sl0 = ch * (TP / S);
#pragma unroll
        for (int j = 0; j < PER; j++) {
            const int i = tid + j * NT;
            const int64_t idx = (int64_t)min(sl0 + i / TV, n_slices - 1) * a.ws_stride +
                                (int64_t)min(v0 + i % TV, V - 1) * S;
            fv[j] = __builtin_nontemporal_load(reinterpret_cast<const v2i64 *>(a.ftl + idx));
            bv[j] = __builtin_nontemporal_load(reinterpret_cast<const v2i64 *>(a.bll + idx));
        }
    };
    load(0);
    for (int32_t ch = 0; ch < n_chunks; ch++) {
        __syncthreads();   // the tiles are free (and s_ord, s_comp, s_bits are set)
#pragma unroll
        for (int j = 0; j < PER; j++) {
            const int i = tid + j * NT, sl = i / TV, r = i % TV;
            t_tl[r][sl * S] = EL::val(fv[j].x, a.lb) - s_comp[r];
            t_tl[r][sl * S + 1] = EL::val(fv[j].y, a.lb) - s_comp[r];
            t_bl[r][sl * S] = EL::val(bv[j].x, a.lb) >> bfo;
            t_bl[r][sl * S + 1] = EL::val(bv[j].y, a.lb) >> bfo;
        }
        if (ch + 1 < n_chunks) load(ch + 1);
        const int32_t p = ch * TP + 2 * lane;   // this lane's two placement columns
        const int64_t m0 = a.makespan[min(p, P - 1)], m1 = a.makespan[min(p + 1, P - 1)];
        __syncthreads();
        BW bits0 = 0, bits1 = 0;
        if (p < P) {
#pragma unroll
            for (int k = 0; k < RPW; k++) {
                const int r = w + k * NW;
                if (v0 + r >= V) continue;
                const int64_t o = (int64_t)s_ord[r] * P + p;
                const long long t0 = t_tl[r][2 * lane], t1 = t_tl[r][2 * lane + 1];
                const long long b0 = t_bl[r][2 * lane], b1 = t_bl[r][2 * lane + 1];
                const bool c0 = t0 + b0 == m0, c1 = t1 + b1 == m1;
                bits0 |= (BW)c0 << r;
                bits1 |= (BW)c1 << r;
                if (even && p + 1 < P) {
                    // written once and streamed past the caches; the flag
                    // pairs stay ordinary stores so that partial lines merge
                    if (a.tl_out) __builtin_nontemporal_store(v2i64{t0, t1}, reinterpret_cast<v2i64 *>(a.tl_out + o));
                    if (a.bl_out) __builtin_nontemporal_store(v2i64{b0, b1}, reinterpret_cast<v2i64 *>(a.bl_out + o));
                    if (crit)
                        *reinterpret_cast<uint16_t *>(crit + o) = (uint16_t)((uint16_t)c0 | ((uint16_t)c1 << 8));
                } else {
                    if (a.tl_out) __builtin_nontemporal_store(t0, &a.tl_out[o]);
                    if (a.bl_out) __builtin_nontemporal_store(b0, &a.bl_out[o]);
                    if (crit) crit[o] = (uint8_t)c0;
                    if (p + 1 < P) {
                        if (a.tl_out) __builtin_nontemporal_store(t1, &a.tl_out[o + 1]);
                        if (a.bl_out) __builtin_nontemporal_store(b1, &a.bl_out[o + 1]);
                        if (crit) crit[o + 1] = (uint8_t)c1;
                    }
                }
            }
        }
        if (cbits != nullptr) {
            __hip_atomic_fetch_or(&s_bits[2 * lane], bits0, __ATOMIC_RELAXED,
                                  __HIP_MEMORY_SCOPE_WORKGROUP);
            __hip_atomic_fetch_or(&s_bits[2 * lane + 1], bits1, __ATOMIC_RELAXED,
                                  __HIP_MEMORY_SCOPE_WORKGROUP);
            __syncthreads();
            if (tid < TP) {
                const int32_t q = ch * TP + tid;
                if (q < P) {
                    const BW x = s_bits[tid];
                    uint32_t *row = cbits + (int64_t)q * n_words + bx * (TV / 32);
                    row[0] = (uint32_t)x;
                    if (TV == 64 && bx * 2 + 1 < n_words) row[1] = (uint32_t)((uint64_t)x >> 32);
                }
                s_bits[tid] = 0;
            }
        }
    }
}

// One wave per placement extracts its canonical critical path. Every path
// node is critical, so the wave (1) lists the placement's critical nodes in
// level-major order from the bit words the emit pass wrote, and (2) maps the
// successor link (an original id) of each listed node to a level-major id.
// When each listed node links to the next one and the last has no successor
// -- no other critical path crosses this one, the usual case -- the list is
// the path, and (2) has already written it out. Otherwise (3) a walk from the
// start follows the links, stepping forward through the sorted list; nodes
// skipped on the way lie on other critical paths. Steps (1) and (2) have no
// dependence between iterations, so many loads are in flight at once; the
// walk reads the lists through registers, 64 x kChaseRegs entries at a time.
// The list lives in the placement's half of its slice of the t workspace,
// which holds nothing needed once the outputs have been emitted; the path is
// written in original ids.
template <int S>
__device__ void chase_wave(const SweepArgs &a, const uint32_t *cbits, int32_t p, int32_t *path,
                           int32_t stride, int32_t *path_len) {
    constexpr int RW = kChaseRegs;
    constexpr int WIN = RW * kWave;
    constexpr int U = 16;  // independent iterations in flight
    const int lane = lane_id();
    const int32_t V = a.V;
    const int32_t slice = p / S, s = p % S;
    const int32_t n_words = (V + 31) / 32;
    // successor links: the low bits of the packed b values, or nx_w (always
    // where the sweep that ran is the gated call's unpacked alternative)
    const bool folded = a.nxf && (a.gate == nullptr || *a.gate == a.gate_want);
    const int32_t *nx = folded ? nullptr : a.nx_w + (int64_t)slice * a.ws_stride;
    const int64_t *bvals = folded ? a.bll + (int64_t)slice * a.ws_stride : nullptr;
    const long long omax = (1ll << a.ob) - 1;
    const uint32_t *bits = cbits + (int64_t)p * n_words;
    // scratch: pos[0, V) and link[V, 2V) in int32 units, in the placement's
    // share of the t workspace (4 ws_stride / S >= 4 (V + pad) int32 each)
    int32_t *pos = reinterpret_cast<int32_t *>(a.ftl) + (int64_t)p * (4 * a.ws_stride / S);
    int32_t *link = pos + V;
    int32_t *out = path + (int64_t)p * stride;
    const int32_t start = __builtin_amdgcn_readfirstlane(a.start[p]);

    // (1) critical nodes in level-major order
    int32_t n = 0;
    for (int32_t w0 = 0; w0 < n_words; w0 += U * kWave) {
        uint32_t wd[U];
#pragma unroll
        for (int j = 0; j < U; j++) {
            const int32_t w = w0 + j * kWave + lane;
            wd[j] = w < n_words ? bits[w] : 0u;
        }
#pragma unroll
        for (int j = 0; j < U; j++) {
            const int32_t cnt = __popc(wd[j]);
            const int32_t incl = wave_incl_scan_i32(cnt);
            int32_t k = n + incl - cnt;
            uint32_t x = wd[j];
            while (x) {
                const int b = __ffs(x) - 1;
                x &= x - 1;
                pos[k++] = 32 * (w0 + j * kWave + lane) + b;
            }
            n += __builtin_amdgcn_readlane(incl, kWave - 1);
        }
    }
    __builtin_amdgcn_s_waitcnt(0);
    // (2) links -> level-major ids (rank[V] = -1: none); the list as the path
    bool chain = n > 0 && start >= 0;
    for (int32_t i0 = 0; i0 < n; i0 += U * kWave) {
        int32_t q[U], qn[U], l[U], o[U];
#pragma unroll
        for (int j = 0; j < U; j++) {
            const int32_t i = min(i0 + j * kWave + lane, n - 1);
            q[j] = pos[i];
            qn[j] = i + 1 < n ? pos[i + 1] : -1;
        }
#pragma unroll
        for (int j = 0; j < U; j++) {
            if (bvals != nullptr) {
                const int64_t t = (bvals[(int64_t)q[j] * S + s] >> a.lb) & omax;
                l[j] = t == 0 ? -1 : (int32_t)(omax - t);
            } else {
                l[j] = nx[(int64_t)q[j] * S + s];
            }
        }
#pragma unroll
        for (int j = 0; j < U; j++) {
            l[j] = a.rank[l[j] < 0 ? V : l[j]];
            o[j] = a.order[q[j]];
        }
#pragma unroll
        for (int j = 0; j < U; j++) {
            const int32_t i = i0 + j * kWave + lane;
            if (i < n) {
                link[i] = l[j];
                // a chain is at most L <= stride long; a longer list is no chain
                if (i < stride) out[i] = o[j];
                chain = chain && l[j] == qn[j] && (i > 0 || q[j] == start);
            }
        }
    }
    chain = __ballot(!chain) == 0ull;
    if (chain || n == 0 || start < 0) {
        if (lane == 0) path_len[p] = start < 0 ? 0 : n;
        return;
    }
    __builtin_amdgcn_s_waitcnt(0);
    // (3) the walk, through register windows of the two lists
    int32_t pa[RW], la[RW], pb[RW], lb[RW];
    auto load = [&](int32_t base, int32_t(&pp)[RW], int32_t(&ll)[RW]) {
#pragma unroll
        for (int j = 0; j < RW; j++) {
            const int32_t i = min(base + j * kWave + lane, n - 1);
            pp[j] = pos[i];
            ll[j] = link[i];
        }
    };
    int32_t c = start;
    int32_t len = 0, acc = -1, i = 0, wb = 0;
    bool going = true;
    load(0, pa, la);
    load(WIN, pb, lb);
    auto walk = [&](int32_t(&pp)[RW], int32_t(&ll)[RW]) {
        if (!going) return;
        // entries [wb, wb + WIN) are in pp / ll; the next window is in flight
        while (i < wb + WIN && i < n) {
            const int32_t x = i - wb;
            const int32_t q = __builtin_amdgcn_readlane(pp[x / kWave], x & (kWave - 1));
            i++;
            if (q < c) continue;   // a critical node off this path
            if (q != c) {          // cannot happen: every link names a listed node
                going = false;
                return;
            }
            acc = lane == (len & (kWave - 1)) ? c : acc;
            len++;
            if ((len & (kWave - 1)) == 0) out[len - kWave + lane] = acc;
            c = __builtin_amdgcn_readlane(ll[x / kWave], x & (kWave - 1));
            if (c < 0) {
                going = false;
                return;
            }
        }
        if (i >= n) {
            going = false;
            return;
        }
        wb += WIN;
        load(wb + WIN, pp, ll);   // the walked buffers take the window after next
    };
    while (going) {
        walk(pa, la);
        walk(pb, lb);
    }
    const int32_t r = len & (kWave - 1);
    if (lane < r) out[len - r + lane] = acc;
    __builtin_amdgcn_s_waitcnt(0);
    // level-major ids -> original ids, in place (each lane rewrites what it wrote)
    for (int32_t i0 = 0; i0 < len; i0 += U * kWave) {
        int32_t t[U];
#pragma unroll
        for (int j = 0; j < U; j++) t[j] = i0 + j * kWave + lane < len ? out[i0 + j * kWave + lane] : 0;
#pragma unroll
        for (int j = 0; j < U; j++) t[j] = a.order[t[j]];
#pragma unroll
        for (int j = 0; j < U; j++)
            if (i0 + j * kWave + lane < len) out[i0 + j * kWave + lane] = t[j];
    }
    if (lane == 0) path_len[p] = len;
}

// After the sweeps: the output rows and the critical bit words are emitted
// (bandwidth-bound, many waves), then one wave per placement extracts its
// critical path (latency-bound, few waves).
template <int S>
__global__ __launch_bounds__(256) void k_chase(SweepArgs a, const uint32_t *cbits, int32_t *path,
                                               int32_t stride, int32_t *path_len) {
    const int32_t p = __builtin_amdgcn_readfirstlane(blockIdx.x * (256 / kWave) + wave_id());
    if (p < a.P) chase_wave<S>(a, cbits, p, path, stride, path_len);
}

template <int S, bool PACKED>
__global__ __launch_bounds__(256) void k_emit(SweepArgs a, uint8_t *crit, uint32_t *cbits) {
    __shared__ __align__(16) char smem[emit_lds<kEmitNodes, kEmitCols>()];
    if (a.gate != nullptr && *a.gate != a.gate_want) return;
    if constexpr (S == 2 && PACKED)
        emit_rows_pair<kEmitNodes, kEmitCols>(a, crit, cbits, xcd_major(blockIdx.x, gridDim.x), smem);
    else
        emit_rows<S, PACKED, kEmitNodes, kEmitCols>(a, crit, cbits,
                                                    xcd_major(blockIdx.x, gridDim.x), smem);
}

constexpr int kSingleThreads = 512;
constexpr int kSingleAcc = 768;
constexpr int kBatchThreads = 256;
constexpr int kBatchAcc = 256;

}  // namespace

hipError_t launch_permute_labels(const Graph &g, const int32_t *placement, int32_t *lab_lm) {
    return launch_permute_labels_batch(g, placement, 1, 1, lab_lm, g.V);
}

hipError_t launch_permute_labels_batch(const Graph &g, const int32_t *placements, int32_t P,
                                       int32_t S, int32_t *lab_w, int64_t lab_stride, int32_t K,
                                       int32_t *err, int32_t *fit, uint32_t fit_limit,
                                       bool lab16, const int32_t *gate, int32_t gate_want) {
    if (lab16 && S != kBatchSlots) return hipErrorInvalidValue;
    if (g.V == 0 || P == 0) return hipSuccess;
    dim3 grid((g.V + 63) / 64, (P + 63) / 64);
    if (S == 1)
        k_permute_labels<1><<<grid, 256, 0, g.stream>>>(g.V, P, g.order, placements, lab_w,
                                                        lab_stride, K, err, fit, fit_limit, 0,
                                                        gate, gate_want);
    else if (S == kBatchSlots)
        k_permute_labels<kBatchSlots><<<grid, 256, 0, g.stream>>>(
            g.V, P, g.order, placements, lab_w, lab_stride, K, err, fit, fit_limit, lab16 ? 1 : 0,
            gate, gate_want);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

namespace {

// flag = 0 if some label lies outside [0, limit) (flag set to 1 beforehand)
__global__ void k_label_fit(int32_t V, const int32_t *lab, int32_t limit, int32_t *flag) {
    for (int32_t v = blockIdx.x * blockDim.x + threadIdx.x; v < V; v += gridDim.x * blockDim.x)
        if ((uint32_t)lab[v] >= (uint32_t)limit) *flag = 0;
}

}  // namespace

hipError_t launch_label_fit(const Graph &g, const int32_t *labels, int32_t limit, int32_t *flag) {
    hipError_t e = launch_fill_i32(flag, 1, 1, g.stream);
    if (e != hipSuccess || g.V == 0) return e;
    int64_t blocks = (g.V + 255) / 256;
    k_label_fit<<<(unsigned)(blocks < 4096 ? blocks : 4096), 256, 0, g.stream>>>(g.V, labels,
                                                                               limit, flag);
    return hipGetLastError();
}

hipError_t launch_sweep(const SweepArgs &a, int32_t S, hipStream_t s) {
    const int32_t n_slices = (a.P + S - 1) / S;
    if (n_slices == 0) return hipSuccess;
    if (a.nxf) return hipErrorInvalidValue;   // this sweep stores links in nx_w only
    const bool packed = a.lb > 0;
    if (S == 1 && !packed) {
        constexpr size_t lds = sweep_lds_bytes<1, kSingleAcc, false>();
        k_sweep<1, kSingleThreads, kSingleAcc, false><<<2 * n_slices, kSingleThreads, lds, s>>>(a);
    } else if (S == kBatchSlots && packed) {
        constexpr size_t lds = sweep_lds_bytes<kBatchSlots, kBatchAcc, true>();
        k_sweep<kBatchSlots, kBatchThreads, kBatchAcc, true>
            <<<2 * n_slices, kBatchThreads, lds, s>>>(a);
    } else if (S == kBatchSlots && !packed) {
        constexpr size_t lds = sweep_lds_bytes<kBatchSlots, kBatchAcc, false>();
        k_sweep<kBatchSlots, kBatchThreads, kBatchAcc, false>
            <<<2 * n_slices, kBatchThreads, lds, s>>>(a);
    } else {
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_finish(const SweepArgs &a, int32_t S, uint8_t *crit, uint32_t *cbits,
                         int32_t *path, int32_t stride, int32_t *path_len, hipStream_t s,
                         const SweepArgs *alt) {
    if (a.P == 0) return hipSuccess;
    // S = 1: outputs only (one placement from the pair sweep), no path
    if (S != kBatchSlots && !(S == 1 && path == nullptr && a.lb > 0)) return hipErrorInvalidValue;
    if (path != nullptr && cbits == nullptr) return hipErrorInvalidValue;
    if (alt != nullptr && (S != kBatchSlots || alt->gate == nullptr || a.gate == nullptr))
        return hipErrorInvalidValue;
    if (a.V > 0) {
        const unsigned blocks = (unsigned)((a.V + kEmitNodes - 1) / kEmitNodes);
        uint32_t *bits = path != nullptr ? cbits : nullptr;
        for (const SweepArgs *x : {&a, alt}) {
            if (x == nullptr) continue;
            if (S == 1)
                k_emit<1, true><<<blocks, 256, 0, s>>>(*x, crit, bits);
            else if (x->lb > 0)
                k_emit<kBatchSlots, true><<<blocks, 256, 0, s>>>(*x, crit, bits);
            else
                k_emit<kBatchSlots, false><<<blocks, 256, 0, s>>>(*x, crit, bits);
            const hipError_t e = hipGetLastError();
            if (e != hipSuccess) return e;
        }
    }
    if (path != nullptr) {
        k_chase<kBatchSlots><<<(unsigned)((a.P + 3) / 4), 256, 0, s>>>(a, cbits, path, stride,
                                                                      path_len);
        return hipGetLastError();
    }
    return hipSuccess;
}

}  // namespace pardnn
