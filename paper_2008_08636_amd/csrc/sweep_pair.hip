// sweep_pair.hip -- batched t-level / b-level sweeps (paper Table 2; Alg. 1
// compute_weighted_levels) over many placements of one graph.
//
//   tl(v) = max over in-edges (u,v) of tl(u) + comp(u) + c(u,v)     (0 if none)
//   bl(v) = comp(v) + max over out-edges (v,s) of c(v,s) + bl(s)     (comp(v) if none)
//   c(u,v) = 0 when both ends carry the same label, else edge_cost  (Fig. 2
//            caption: communication inside a cluster counts as zero)
//
// Design for gfx950. A sweep is a chain of L dependent level steps. One
// workgroup of TWO waves walks one chain for S placements, with ONE barrier
// per level:
//   wave 0 ("near"): finalises level i from its LDS accumulators (value, label
//     sums, successor), writes the values to an LDS ring and the workspace,
//     then folds the span-1 edges of level i + 1 -- whose neighbours it has
//     just finalised -- into the accumulators of level i + 1;
//   wave 1 ("far"):  meanwhile folds the longer edges of level i + 1, whose
//     neighbours were final one or more barriers ago: from the LDS ring when
//     they finished in the last D levels, else from registers loaded D levels
//     ahead.
// So the dependent path of a level is one LDS round trip for the
// accumulators, one for the ring, the arithmetic and one barrier; the global
// loads all run ahead:
//   near wave: node constants, labels and span-1 edge records LN levels ahead;
//   far wave:  edge records D + RF levels ahead, neighbour values D ahead.
// Long edges (the neighbour finished well before the owner's block of
// kLongBlock levels begins) read their values from LDS too: per block, the
// far wave gathers the block's distinct long-edge neighbours, sorted by
// position, one 64-lane chunk per level, into one of two LDS buffers ahead of
// the block. Neighbours that several nearby levels share then cost one
// gather, and neighbours on one cache line one line request: the per-level
// gathers that remain are the few edges of medium span.
// The register state of the levels in flight rotates by name through an
// NS-times unrolled loop, and every global load and store of a fast level is
// unconditional (clamped addresses; idle lanes store into the slice's
// padding), so the in-order wait counters never drain the pipeline.
//
// The b keys carry the successor tie-break in their low bits,
// (value << ob) | (2^ob - 1 - successor's original id), so the maximum names
// the canonical successor. Levels outside the fast shape (more than 64
// nodes, 64 * kNEn span-1 edges or 64 * kNEf longer edges) take a general
// path that drains the workgroup, processes the level in chunks from the
// workspace, and refills the pipeline.
#include "device_utils.h"
#include "internal.h"
#include "sweep_common.h"

#include <algorithm>
#include <utility>

namespace pardnn {

namespace {

constexpr int kLanes = 64;
constexpr int kPNodes = 64;          // nodes of a fast level, one per lane of wave 0
constexpr int kNEn = 2;              // span-1 edge tasks per lane of wave 0
constexpr int kNEf = 3;              // longer-edge tasks per lane of wave 1
constexpr int kD = 3;                // far values loaded D levels ahead
constexpr int kRF = 3;               // far records loaded RF levels before their values
constexpr int kNS = kD + kRF + 2;    // register sets in flight (loop unrolling)
constexpr int kLN = kNS - 2;         // wave 0 loads LN levels ahead
constexpr int kRS = kD + 1;          // LDS ring slots (levels)
constexpr int kNB = 8;               // accumulator buffers (levels; >= kD + 2, a power of 2)
static_assert(kNB >= kD + 2 && (kNB & (kNB - 1)) == 0, "accumulator buffers");
constexpr int kPBinsCap = 2048;      // labels x slots of the LDS label bins
// long edges: the ring's LDS entries are followed by two bulk buffers of
// kLongCap entries; a block is one unrolled group of levels
static_assert(kLongBlock == kNS, "one long-edge block per unrolled group");
static_assert(kLongCap == kLongBlock * kLanes, "one 64-lane chunk per level of a block");
static_assert(kLongBase == (uint32_t)(kRS * kPNodes), "bulk buffers follow the ring");
static_assert(kLongBase + 2 * kLongCap <= kPreFolded, "ring field range");
// chunk c of block k is listed at step 8k - 14 + c, gathered at 8k - 11 + c
// and stored to LDS at 8k - 9 + c; the block is read from step 8k - 1 (the
// far folds of its first level) to 8k + 6. Its neighbours must be final when
// gathered: finished by step 8k - 12.
static_assert(kLongLead >= kLongBlock + 4, "long neighbours final when gathered");
// label sums of the t sweep: none, in LDS bins (K S <= kPBinsCap), or by
// global atomics; a template parameter, so that a chain carries one of them
constexpr int kBinsNone = 0, kBinsLds = 1, kBinsGlobal = 2;

typedef const __attribute__((address_space(4))) PairLevel *ConstPairLevel;
typedef const __attribute__((address_space(4))) SweepArgs KArgs;
typedef __attribute__((address_space(3))) char LdsBytes;   // the dynamic LDS, as bytes

// The kernel's argument block (its only argument, at offset 0 of the kernarg
// segment) through a pointer the compiler cannot see through, so that loads
// from it stay where they are written: the general level path re-reads its
// pointers instead of the loop keeping them live. Defined in the kernel's own
// code only (a called function would read a null segment pointer).
__device__ __forceinline__ KArgs *kargs_here() {
    KArgs *p = (KArgs *)__builtin_amdgcn_kernarg_segment_ptr();
    asm volatile("" : "+s"(p));
    return p;
}

template <int I>
struct IC {
    static constexpr int value = I;
};

// f(IC<0>), ..., f(IC<kNS - 1>): one group of levels, each with its register
// sets named at compile time
template <class F, int... I>
__device__ __forceinline__ void unroll_seq(F &f, std::integer_sequence<int, I...>) {
    (f(IC<I>{}), ...);
}

// S values / labels of one node (its S placements), adjacent in memory.
template <int S>
struct alignas(S * 8 >= 16 ? 16 : S * 8) VecS {
    int64_t v[S];
};
template <int S>
struct alignas(4 * S >= 16 ? 16 : 4 * S) LabS {
    int32_t v[S];
};

// Level bounds of one step as staged in the LDS window: first node, first
// near and far record, and the three counts saturated at 255 (enough to tell
// a fast level; the general path reads exact bounds).
struct alignas(16) WinEnt {
    int32_t nlo, nrlo, frlo;
    uint32_t cnt;   // min(w,255) | min(near,255) << 8 | min(far,255) << 16 | fast << 31
};
constexpr int kWin = 128;            // window entries (steps); refilled every kWin / 2

__device__ __forceinline__ int32_t cnt_w(uint32_t c) { return (int32_t)(c & 255u); }
__device__ __forceinline__ int32_t cnt_near(uint32_t c) { return (int32_t)((c >> 8) & 255u); }
__device__ __forceinline__ int32_t cnt_far(uint32_t c) { return (int32_t)((c >> 16) & 255u); }
// a level of the fast shape: at most 64 nodes, 64 kNEn span-1 and 64 kNEf
// longer edges, of which at most 64 read the workspace (decided when the
// window entry is staged)
__device__ __forceinline__ bool cnt_fast(uint32_t c) { return (int32_t)c < 0; }

template <int S>
struct NearSet {   // wave 0, one level
    uint32_t ol[kNEn];
    int64_t c[kNEn];
    int64_t comp, mem;
    LabS<S> lab;
    int32_t wnlo;      // the level's first node and counts (its window entry),
    uint32_t wcnt;     // carried with the set instead of re-read at every use
};

template <int S>
struct FarSet {    // wave 1, one level
    int32_t nb[kNEf];
    uint32_t ol[kNEf];
    int64_t c[kNEf];
    VecS<S> f;         // the workspace value of task 0 (only task 0 reads one)
    uint32_t wcnt;     // the level's counts (its window entry)
};

template <int S>
constexpr size_t pair_lds_fixed() {
    return (size_t)kWin * sizeof(WinEnt)        // bounds window
           + (size_t)kNB * kPNodes * S * 8       // acc[kNB]
           + (size_t)kRS * kPNodes * S * 8       // ring
           + (size_t)2 * kLongCap * S * 8        // long-edge buffers (after the ring)
           + (size_t)2 * kPNodes * S * 4;        // slab[2]
}

// Everything a chain derives from the arguments: the slice's workspace, the
// LDS layout and the value encoding. NXF (b only): the successor links ride
// in the b values, a property of the launch fixed at compile time so that
// the b chain carries no arithmetic of the other encoding.
template <int S, bool FWD, int BM, bool NXF>
struct PairCtx {
    static constexpr bool want_bins = FWD && BM != kBinsNone;
    static constexpr bool lds_bins = FWD && BM == kBinsLds;
    using EL = Elem<true>;
    using VS = VecS<S>;
    using LS = LabS<S>;
    // two 16-bit labels per node (every batch: S = 2); a fast level's load
    // keeps the word as it is (in v[0]) until the labels are used, so that
    // nothing waits for the load early
    static constexpr bool L16 = S == 2;
    int lane, tid;
    int32_t V, L, P, K, p0;
    int32_t s0, s1, gen_end;   // steps of this chain; general path before gen_end
    int lb, ob;
    int fo;          // bits of successor link below a workspace value's label (b, folded)
    long long omax;
    VS *vals;
    const void *labs;
    LS *nxs;
    bool want_nx;
    ConstPairLevel pls;
    WinEnt *win;
    long long *acc;
    VS *ring;
    LS *slab;
    long long *bins;

    template <class AP>
    __device__ __forceinline__ PairCtx(AP a, int32_t slice, char *smem) {
        lane = lane_id();
        tid = threadIdx.x;   // 0 .. 127 over both waves
        V = a->V;
        L = a->L;
        s0 = a->seg_on ? (FWD ? a->seg_t0 : a->seg_b0) : 0;
        s1 = a->seg_on ? (FWD ? a->seg_t1 : a->seg_b1) : L;
        gen_end = s0 > 0 ? s0 + kD + 1 : 0;
        P = a->P;
        K = a->K;
        p0 = slice * S;
        lb = a->lb;
        ob = FWD ? 0 : a->ob;
        fo = !FWD && NXF ? ob : 0;
        omax = (1ll << ob) - 1;
        vals = reinterpret_cast<VS *>((FWD ? a->ftl : a->bll) + (int64_t)slice * a->ws_stride);
        labs = L16 ? (const void *)(reinterpret_cast<const uint16_t *>(a->lab_w) +
                                    (int64_t)slice * a->lab_stride)
                   : (const void *)(a->lab_w + (int64_t)slice * a->lab_stride);
        want_nx = !FWD && !NXF && a->nx_w != nullptr;
        nxs = reinterpret_cast<LS *>(a->nx_w + (want_nx ? (int64_t)slice * a->ws_stride : 0));
        pls = (ConstPairLevel)(FWD ? a->pl_t : a->pl_b);
        win = reinterpret_cast<WinEnt *>(smem);                       // [kWin]
        acc = reinterpret_cast<long long *>(win + kWin);              // [kNB][64 S]
        ring = reinterpret_cast<VS *>(acc + kNB * kPNodes * S);       // [kRS][64], [2][kLongCap]
        slab = reinterpret_cast<LS *>(ring + kLongBase + 2 * kLongCap);   // [2][64]
        bins = reinterpret_cast<long long *>(slab + 2 * kPNodes);     // [K S]
    }
    // node v's labels as loaded: the 32-bit labels, or (L16) the word of its
    // two 16-bit labels in v[0]
    __device__ __forceinline__ LS lab_raw(uint32_t v) const {
        LS r;
        if constexpr (L16) {
            r.v[0] = (int32_t)at(reinterpret_cast<const uint32_t *>(labs), v);
            r.v[1] = 0;
        } else {
            r = at(reinterpret_cast<const LS *>(labs), v);
        }
        return r;
    }
    __device__ __forceinline__ LS lab_use(const LS &x) const {
        if constexpr (L16) {
            LS r;
            r.v[0] = (int32_t)((uint32_t)x.v[0] & 0xffffu);
            r.v[1] = (int32_t)((uint32_t)x.v[0] >> 16);
            return r;
        } else {
            return x;
        }
    }
    __device__ __forceinline__ LS lab(uint32_t v) const { return lab_use(lab_raw(v)); }
    // the tl + comp or bl of a workspace (or ring) value
    __device__ __forceinline__ int64_t gval(int64_t g) const {
        if constexpr (!FWD && NXF)
            return EL::val(g, lb) >> ob;
        else
            return EL::val(g, lb);
    }
    __device__ __forceinline__ int64_t cand(int64_t g, int32_t own_lab, int64_t c) const {
        return gval(g) + (EL::lab(g, lb) != own_lab ? c : 0);
    }
    __device__ __forceinline__ long long akey(int64_t cv, int32_t tie) const {
        return FWD ? cv : (cv << ob) | tie;
    }
    // the key of an edge record's candidate from its cost word ck (t: ob = 0)
    __device__ __forceinline__ long long rkey(int64_t g, int32_t own_lab, int64_t ck) const {
        const bool cross = EL::lab(g, lb) != own_lab;
        if constexpr (FWD)
            return gval(g) + (cross ? ck : 0);
        else if constexpr (NXF)   // the value's key bits sit above its link bits already
            return ((g >> lb) & ~omax) + (cross ? ck : (ck & omax));
        else
            return ((g >> lb) << ob) + (cross ? ck : (ck & omax));
    }
    __device__ __forceinline__ int32_t level_of(int32_t step) const {   // L: empty level
        if (FWD) return step < L ? step : L;
        return step < L ? L - 1 - step : L;
    }
    __device__ __forceinline__ WinEnt W(int32_t step) const { return win[step & (kWin - 1)]; }
    __device__ __forceinline__ long long *accb(int32_t step) const {
        return acc + ((uint32_t)step % kNB) * kPNodes * S;
    }

    // finalise node v (slot = its index in the level) from the level's
    // accumulators: value, successor, ring entry, label sums, workspace
    __device__ __forceinline__ void finish(int64_t *label_mem, int32_t step, int32_t v, bool act,
                                           bool to_ring, int slot, int64_t comp, int64_t mem,
                                           const LS &lab, bool side = true) const {
        long long *ab = accb(step);
        VS out;
        long long kk[S];
#pragma unroll
        for (int s = 0; s < S; s++) {
            const long long k = ab[slot * S + s];
            kk[s] = k;
            // b, folded: (comp << ob) + k = ((comp + max) << ob) | successor's tie
            // key, with k = 0 (no successor) leaving the link bits 0
            const int64_t x = FWD ? k + comp : NXF ? (comp << ob) + k : comp + (k >> ob);
            out.v[s] = EL::make(x, lab.v[s], lb);
        }
        if (act && to_ring) ring[((uint32_t)step % kRS) * kPNodes + slot] = out;
        const uint32_t sv = act ? (uint32_t)v : (uint32_t)V;   // idle lanes: one padding slot
        at(vals, sv) = out;
        if (want_nx) {
            LS nxv;
#pragma unroll
            for (int s = 0; s < S; s++)
                nxv.v[s] = kk[s] == 0 ? -1 : (int32_t)(omax - (kk[s] & omax));
            at(nxs, sv) = nxv;
        }
        if (side) finish_side(label_mem, step, act, slot, mem, lab);
    }
    // the parts of finishing a node that nothing reads soon: clearing its
    // accumulator slot and its label sums
    __device__ __forceinline__ void finish_side(int64_t *label_mem, int32_t step, bool act, int slot,
                                                int64_t mem, const LS &lab) const {
        long long *ab = accb(step);
#pragma unroll
        for (int s = 0; s < S; s++) ab[slot * S + s] = 0;
        if (act) {
            if constexpr (want_bins) {
#pragma unroll
                for (int s = 0; s < S; s++) {
                    const int32_t l = lab.v[s];
                    if ((uint32_t)l < (uint32_t)K && p0 + s < P) {
                        if constexpr (lds_bins)
                            lds_add_i64(&bins[l * S + s], mem);
                        else
                            atomicAdd((unsigned long long *)&label_mem[(int64_t)(p0 + s) * K + l],
                                      (unsigned long long)mem);
                    }
                }
            }
        }
    }
};

// First step of the pipelined loop: a multiple of kNS, so that a step's
// register set and LDS slots follow from its position in the unrolled group;
// a segment that starts past step 0 walks its first levels (at least D + 1,
// whose LDS state the walk has not built) on the general path up to it.
template <class Ctx>
__device__ __forceinline__ int32_t pipe_start(const Ctx &c) {
    if (c.s0 == 0) return 0;
    return min(c.s1, (c.gen_end + kNS - 1) & ~(kNS - 1));
}

// The general level step, for both waves: the level in chunks of 64 nodes
// from the workspace, the early folds of a level too wide for the ring, and
// the next level's edges. Everything it reads from the arguments is read
// afresh through `a` (the kernel's argument block: the kernarg segment
// pointer is defined in the kernel only, so the caller passes it), so that the
// pipelined loop around it does not carry its pointers in registers. It is a
// real call, not inlined: the unrolled loop would otherwise hold eight copies
// of it per chain, and the smaller loop body takes instruction-cache misses
// off every fast level.
template <int S, bool FWD, bool NEAR, int BM, bool NXF>
__device__ __attribute__((noinline)) void pair_slow(KArgs *a, int32_t slice, int32_t step,
                                                    LdsBytes *smem_l) {
    char *smem = (char *)smem_l;
    const PairCtx<S, FWD, BM, NXF> c(a, slice, smem);
    using VS = VecS<S>;
    using LS = LabS<S>;
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    const int32_t *offs = FWD ? a->in_off : a->out_off;
    const int32_t *srcs = FWD ? a->in_src : a->out_dst;
    const int32_t *owns = FWD ? a->in_dst : a->out_src;
    const int64_t *costs = FWD ? a->in_cost : a->out_cost;
    const int32_t x = c.level_of(step), xn = c.level_of(step + 1);
    const int32_t lo = c.pls[x].node_lo, hi = c.pls[x + 1].node_lo;
    const bool to_ring = hi - lo <= kPNodes;
    const uint32_t vmax = (uint32_t)(c.V - 1);
    auto fold = [&](int32_t cn0, int32_t cea, int32_t ceb, long long *ab) {
        for (int32_t e = cea + c.tid; e < ceb; e += 2 * kLanes) {
            const int32_t nb = srcs[e], own = owns[e] - cn0;
            const int64_t cost = costs[e];
            const int32_t tie = FWD ? 0 : (int32_t)(c.omax - a->out_dst_orig[e]);
            const VS g = c.vals[nb];
            const LS ol = c.lab(cn0 + own);
#pragma unroll
            for (int s = 0; s < S; s++)
                lds_max_i64(&ab[own * S + s], c.akey(c.cand(g.v[s], ol.v[s], cost), tie));
        }
    };
    for (int32_t cn0 = lo; cn0 < hi; cn0 += kPNodes) {
        const int32_t cn1 = min(hi, cn0 + kPNodes);
        fold(cn0, offs[cn0], offs[cn1], c.accb(step));
        __syncthreads();
        if (NEAR) {
            const int32_t v = cn0 + c.lane;
            const uint32_t vc = min((uint32_t)v, vmax);
            const NodeRec16 nr = at(a->node_rec, vc);
            c.finish(a->label_mem, step, v, v < cn1, to_ring, c.lane, nr.comp, nr.mem, c.lab(vc));
        }
        __syncthreads();
    }
    // a level too wide for the ring: fold its edges of span 2 .. D + 1 now
    // into the accumulators of their (narrow) owners' levels; the far records
    // mark them kPreFolded
    if (!to_ring) {
        const int32_t *poff = FWD ? a->preoff_t : a->preoff_b;
        const PreRec16 *pre = FWD ? a->pre_t : a->pre_b;
        for (int32_t e = poff[x] + c.tid; e < poff[x + 1]; e += 2 * kLanes) {
            const PreRec16 r = pre[e];
            const int32_t own = (int32_t)(r.os & 0xffffu), span = (int32_t)(r.os >> 16);
            const int32_t tie = FWD ? 0 : a->pretie_b[e];
            const VS g = c.vals[r.nb];
            const LS ol = c.lab(c.W(step + span).nlo + own);
            long long *ab = c.accb(step + span);
#pragma unroll
            for (int s = 0; s < S; s++)
                lds_max_i64(&ab[own * S + s], c.akey(c.cand(g.v[s], ol.v[s], r.cost), tie));
        }
    }
    // the next level's edges, all from the workspace (everything before it is
    // final now), unless that level takes this path itself
    if (cnt_fast(c.W(step + 1).cnt)) {
        const int32_t nlo = c.pls[xn].node_lo, nhi = c.pls[xn + 1].node_lo;
        fold(nlo, offs[nlo], offs[nhi], c.accb(step + 1));
    }
}

template <int S, bool FWD, bool NEAR, int BM, bool NXF>
__device__ __forceinline__ void pair_chain(const SweepArgs &a, int32_t slice, char *smem) {
    using EL = Elem<true>;
    using VS = VecS<S>;
    using LS = LabS<S>;
    const PairCtx<S, FWD, BM, NXF> c(&a, slice, smem);
    const int lane = c.lane;
    const int32_t L = c.L;
    const uint32_t vmax = c.V > 0 ? (uint32_t)(c.V - 1) : 0u;
    const PairLevel *plv = FWD ? a.pl_t : a.pl_b;   // per-lane reads

    // the window entry of step sx from its level's bounds l0, l1
    auto fill_entry = [&](int32_t sx, const PairLevel &l0, const PairLevel &l1) {
            WinEnt e;
            e.nlo = l0.node_lo;
            e.nrlo = l0.near_lo;
            e.frlo = l0.far_lo;
            const int32_t w = l1.node_lo - l0.node_lo, nn = l1.near_lo - l0.near_lo,
                          nf = l1.far_lo - l0.far_lo;
            const bool fast = w <= kPNodes && nn <= kNEn * kLanes && nf <= kNEf * kLanes &&
                              l0.n_gather <= kLanes && sx >= c.gen_end;
            e.cnt = (uint32_t)min(w, 255) | (uint32_t)min(nn, 255) << 8 |
                    (uint32_t)min(nf, 255) << 16 | (fast ? 1u << 31 : 0u);
            c.win[sx & (kWin - 1)] = e;
    };
    // window entries for steps s0 + lane + 64 k, k < n (wave 0, synchronous:
    // before the pipelined loop)
    auto fill = [&](int32_t s0, int n) {
        for (int k = 0; k < n; k++) {
            const int32_t sx = s0 + lane + k * kLanes;
            const int32_t x = c.level_of(sx);
            fill_entry(sx, plv[x], plv[x + 1]);
        }
    };

    if (NEAR) {
        // ================= wave 0: finalise + span-1 edges =================
        const NearRec12 *nrec = FWD ? a.nr_t : a.nr_b;
        NearSet<S> st[kNS];
        // unconditional loads (idle lanes read element 0), so that the
        // compiler's in-order wait counts are the same on every path
        auto loads = [&](NearSet<S> &X, const WinEnt &b) {
            const int32_t nn = cnt_near(b.cnt), w = cnt_w(b.cnt);
#pragma unroll
            for (int j = 0; j < kNEn; j++) {
                const uint32_t e = lane + j * kLanes < nn ? (uint32_t)(b.nrlo + lane + j * kLanes) : 0u;
                const NearRec12 r = at(nrec, e);
                X.ol[j] = r.ol;
                X.c[j] = (int64_t)(((uint64_t)r.ck_hi << 32) | r.ck_lo);
            }
            const uint32_t v = lane < w ? (uint32_t)(b.nlo + lane) : 0u;
            if constexpr (FWD && BM != kBinsNone) {   // the label sums need the memory
                const NodeRec16 n = at(a.node_rec, v);
                X.comp = n.comp;
                X.mem = n.mem;
            } else {
                X.comp = at(a.comp_lm, v);
                X.mem = 0;
            }
            X.lab = c.lab_raw(v);
            X.wnlo = b.nlo;
            X.wcnt = b.cnt;
        };
        // after level `step`: labels of step + 2, loads of step + LN, window refill
        // the window is refilled 64 entries at a time, 64 steps ahead: the
        // bounds load at step 64 m and the entries go to LDS at step 64 m + 4,
        // so the stores wait on loads that are due by then anyway (a
        // synchronous refill drained every load in flight)
        PairLevel fl0 = {}, fl1 = {};
        auto tail = [&](int32_t step, const NearSet<S> &B2, NearSet<S> &LD, const WinEnt &b2,
                        const WinEnt &bl) {
            loads(LD, bl);
            if ((step & (kWin / 2 - 1)) == 0 && step > 0) {
                const int32_t x = c.level_of(step + kWin / 2 + lane);
                fl0 = plv[x];
                fl1 = plv[x + 1];
            }
            if ((step & (kWin / 2 - 1)) == 4 && step > 4) fill_entry(step - 4 + kWin / 2 + lane, fl0, fl1);
            __syncthreads();
        };
        auto body = [&](int32_t step, const WinEnt &b0, const WinEnt &b1, NearSet<S> &A,
                        const NearSet<S> &B1) {
            c.finish(a.label_mem, step, b0.nlo + lane, lane < cnt_w(b0.cnt), true, lane, A.comp, A.mem,
                     c.lab_use(A.lab), false);
            // span-1 edges of the next level, from the ring slot just written
            if (cnt_fast(b1.cnt)) {
                const int32_t nt = cnt_near(b1.cnt);
                long long *ab = c.accb(step + 1);
                const LS *sl = c.slab + ((step + 1) & 1) * kPNodes;
                const VS *rs = c.ring + ((uint32_t)step % kRS) * kPNodes;
#pragma unroll
                for (int j = 0; j < kNEn; j++) {
                    if (lane + j * kLanes < nt) {
                        const uint32_t own = B1.ol[j] & 0xffffu, nbl = B1.ol[j] >> 16;
                        const VS g = rs[nbl];
                        const LS ol = sl[own];
#pragma unroll
                        for (int s = 0; s < S; s++)
                            lds_max_i64(&ab[own * S + s], c.rkey(g.v[s], ol.v[s], B1.c[j]));
                    }
                }
            }
            // after the folds, so that the LDS (in order) serves the folds'
            // reads first
            c.finish_side(a.label_mem, step, lane < cnt_w(b0.cnt), lane, A.mem, c.lab_use(A.lab));
        };
        const int32_t s0 = c.s0, s1 = c.s1;
        const int32_t a0 = pipe_start(c);
        if (s1 > s0) {
            fill(s0, kWin / kLanes);
            for (int i = lane; i < kNB * kPNodes * S; i += kLanes) c.acc[i] = 0;
            if (c.lds_bins)
                for (int i = lane; i < c.K * S; i += kLanes) c.bins[i] = 0;
            __builtin_amdgcn_s_waitcnt(0);
        }
        __syncthreads();
        // the window entry of the level each step loads, read one step ahead
        WinEnt wn[2];
        // a segment's first levels, on the general path
        for (int32_t sx = s0; sx < a0; sx++) {
            pair_slow<S, FWD, true, BM, NXF>(kargs_here(), c.p0 / S, sx, (LdsBytes *)c.win);
            __syncthreads();
        }
        if (a0 < s1) {
#pragma unroll
            for (int j = 0; j < kLN; j++) loads(st[j], c.W(a0 + j));
            __builtin_amdgcn_s_waitcnt(0);
            if (lane < cnt_w(c.W(a0 + 1).cnt)) c.slab[((a0 + 1) & 1) * kPNodes + lane] = c.lab_use(st[1].lab);
            wn[0] = c.W(a0 + kLN);
        }
        __syncthreads();
        int32_t step = a0;
        auto one = [&](auto RC) {
            constexpr int r = decltype(RC)::value;
            if constexpr (r < kNS) {
                // step == r modulo kNS here; written so that the compiler sees
                // it, and the LDS slots of the step become constants
                const int32_t sa = (int32_t)(((uint32_t)step & ~(uint32_t)(kNS - 1)) | (uint32_t)r);
                // the entries of levels step .. step + 2 came with their sets;
                // only the one of the level loaded now is read from LDS
                const WinEnt b0 = {st[r].wnlo, 0, 0, st[r].wcnt};
                const WinEnt b1 = {0, 0, 0, st[(r + 1) % kNS].wcnt};
                const WinEnt b2 = {0, 0, 0, st[(r + 2) % kNS].wcnt};
                // off the level's dependent LDS chain: the labels of level
                // step + 2 (their slot was last read at the step before) and
                // the window entry the next step's loads need
                if (lane < cnt_w(b2.cnt)) c.slab[(sa & 1) * kPNodes + lane] = c.lab_use(st[(r + 2) % kNS].lab);
                const WinEnt bl = wn[r & 1];
                {
                    // an index the compiler cannot see is zero: the entry
                    // stays in vector registers and nothing waits for it
                    // before its first use
                    int32_t z;
                    asm volatile("v_mov_b32 %0, 0" : "=v"(z));
                    wn[(r + 1) & 1] = c.win[((sa + kLN + 1) & (kWin - 1)) + z];
                }
                if (cnt_fast(b0.cnt))
                    body(sa, b0, b1, st[r], st[(r + 1) % kNS]);
                else
                    pair_slow<S, FWD, true, BM, NXF>(kargs_here(), c.p0 / S, sa, (LdsBytes *)c.win);
                tail(sa, st[(r + 2) % kNS], st[(r + kLN) % kNS], b2, bl);
                step++;
            }
        };
        // whole groups of kNS levels only: an exit inside the unrolled group
        // would merge every body's loads in flight into the loop header
        while (step + kNS <= s1) unroll_seq(one, std::make_integer_sequence<int, kNS>{});
        // the last levels (fewer than kNS) on the general path; folding an
        // edge a second time into a maximum changes nothing
        for (; step < s1; step++) {
            pair_slow<S, FWD, true, BM, NXF>(kargs_here(), c.p0 / S, step, (LdsBytes *)c.win);
            __syncthreads();
        }
    } else {
        // ================= wave 1: longer edges =================
        const FarRec16 *frec = FWD ? a.fr_t : a.fr_b;
        FarSet<S> st[kNS];
        auto records = [&](FarSet<S> &X, const WinEnt &b) {
            const int32_t nf = cnt_far(b.cnt);
            X.wcnt = b.cnt;
#pragma unroll
            for (int j = 0; j < kNEf; j++) {
                // tasks past the level's records are never read: load them
                // only where the level has records for them (uniform)
                if (j > 0 && nf <= j * kLanes) continue;
                const uint32_t e = lane + j * kLanes < nf ? (uint32_t)(b.frlo + lane + j * kLanes) : 0u;
                const FarRec16 r = at(frec, e);
                X.nb[j] = r.nb;
                X.ol[j] = r.ol;
                X.c[j] = r.ck;
            }
        };
        // a fast level's records that read the workspace come first, at
        // most 64 of them: task 0 of each lane
        auto far_loads = [&](FarSet<S> &X, const WinEnt &b) {
            const bool far = lane < cnt_far(b.cnt) && (X.ol[0] >> 16) == kNoRing;
            X.f = at(c.vals, far ? (uint32_t)X.nb[0] : 0u);
        };
        auto fold_far = [&](int32_t step, const FarSet<S> &B1, const WinEnt &b1) {
            const int32_t nt = cnt_far(b1.cnt);
            long long *ab = c.accb(step + 1);
            const LS *sl = c.slab + ((step + 1) & 1) * kPNodes;
#pragma unroll
            for (int j = 0; j < kNEf; j++) {
                if (lane + j * kLanes < nt && (B1.ol[j] >> 16) != kPreFolded) {
                    const uint32_t own = B1.ol[j] & 0xffffu, rg = B1.ol[j] >> 16;
                    const VS g = j == 0 && rg == kNoRing ? B1.f : c.ring[rg];
                    const LS ol = sl[own];
#pragma unroll
                    for (int s = 0; s < S; s++)
                        lds_max_i64(&ab[own * S + s], c.rkey(g.v[s], ol.v[s], B1.c[j]));
                }
            }
        };
        // long edges, step i (position r = i mod kNS): list chunk (r + 6) mod
        // 8, gather chunk (r + 3) mod 8 (listed three steps ago), store chunk
        // (r + 1) mod 8 (gathered two steps ago); lst and lval rotate by name
        const int32_t *lsrc = FWD ? a.lsrc_t : a.lsrc_b;
        VS *lbuf = c.ring + kLongBase;
        // (values as plain elements: whole-record copies would stay in
        // scratch memory)
        int32_t lst[4];
        int64_t lval[4][S];
        auto long_entry = [&](int32_t k, int ch) {
            return at(lsrc, (uint32_t)(k * kLongCap + ch * kLanes + lane));
        };
        auto long_load = [&](int64_t(&d)[S], int32_t v) {
            const VS &g = at(c.vals, (uint32_t)v);
#pragma unroll
            for (int s = 0; s < S; s++) d[s] = g.v[s];
        };
        auto long_put = [&](int32_t k, int ch, const int64_t(&x)[S]) {
            VS &d = lbuf[(k & 1) * kLongCap + ch * kLanes + lane];
#pragma unroll
            for (int s = 0; s < S; s++) d.v[s] = x[s];
        };
        auto long_list = [&](int32_t i, auto RC) {
            constexpr int r = decltype(RC)::value, ch = (r + 6) % kLongBlock;
            lst[r % 4] = long_entry((i + 14 - ch) / kLongBlock, ch);
        };
        auto long_gather = [&](auto RC) {
            constexpr int r = decltype(RC)::value;
            long_load(lval[r % 4], lst[(r + 1) % 4]);
        };
        auto long_store = [&](int32_t i, auto RC) {
            constexpr int r = decltype(RC)::value, ch = (r + 1) % kLongBlock;
            long_put((i + 9 - ch) / kLongBlock, ch, lval[(r + 2) % 4]);
        };
        __syncthreads();   // the window is filled by wave 0
        const int32_t s0 = c.s0, s1 = c.s1;
        const int32_t a0 = pipe_start(c);
        for (int32_t sx = s0; sx < a0; sx++) {
            pair_slow<S, FWD, false, BM, NXF>(kargs_here(), c.p0 / S, sx, (LdsBytes *)c.win);
            __syncthreads();
        }
        if (a0 < s1) {
            // what the long-edge steps before a0 leave behind (a0 is a
            // multiple of kNS, every neighbour they read is final): block b0
            // and the first chunk of block b0 + 1 in LDS, the next two chunks
            // gathered, the three after them listed
            const int32_t b0 = a0 / kLongBlock;
            {
                int32_t l[kLongBlock + 1];
#pragma unroll
                for (int ch = 0; ch < kLongBlock; ch++) l[ch] = long_entry(b0, ch);
                l[kLongBlock] = long_entry(b0 + 1, 0);
                lst[2] = long_entry(b0 + 1, 1);
                lst[3] = long_entry(b0 + 1, 2);
                __builtin_amdgcn_s_waitcnt(0);
                int64_t v[kLongBlock + 1][S];
#pragma unroll
                for (int ch = 0; ch <= kLongBlock; ch++) long_load(v[ch], l[ch]);
                long_load(lval[2], lst[2]);
                long_load(lval[3], lst[3]);
                __builtin_amdgcn_s_waitcnt(0);
#pragma unroll
                for (int ch = 0; ch < kLongBlock; ch++) long_put(b0, ch, v[ch]);
                long_put(b0 + 1, 0, v[kLongBlock]);
                lst[1] = long_entry(b0 + 1, 3);
                lst[2] = long_entry(b0 + 1, 4);
                lst[3] = long_entry(b0 + 1, 5);
            }
            st[0].wcnt = c.W(a0).cnt;
#pragma unroll
            for (int j = 1; j <= kD + kRF; j++) records(st[j], c.W(a0 + j));
            __builtin_amdgcn_s_waitcnt(0);
            // the values of the first levels' distant neighbours (none when
            // the chain starts at level 0)
#pragma unroll
            for (int j = 1; j <= kD; j++) far_loads(st[j], c.W(a0 + j));
            // nothing may be pending at the loop entry: a load in flight into a
            // register the loop reuses would make the loop header wait for it
            __builtin_amdgcn_s_waitcnt(0);
        }
        __syncthreads();
        int32_t step = a0;
        auto one = [&](auto RC) {
            constexpr int r = decltype(RC)::value;
            if constexpr (r < kNS) {
                const int32_t sa = (int32_t)(((uint32_t)step & ~(uint32_t)(kNS - 1)) | (uint32_t)r);
                const WinEnt b0 = {0, 0, 0, st[r].wcnt};
                const WinEnt b1 = {0, 0, 0, st[(r + 1) % kNS].wcnt};
                const WinEnt bd = {0, 0, 0, st[(r + 1 + kD) % kNS].wcnt};
                const WinEnt brf = c.W(sa + 1 + kD + kRF);
                FarSet<S> &B1 = st[(r + 1) % kNS];
                if (cnt_fast(b0.cnt)) {
                    if (cnt_fast(b1.cnt)) fold_far(sa, B1, b1);
                } else {
                    pair_slow<S, FWD, false, BM, NXF>(kargs_here(), c.p0 / S, sa, (LdsBytes *)c.win);
                }
                // the long-edge loads before the step's other loads: the waits
                // they need then fall on loads the steps need anyway
                long_list(sa, RC);
                long_gather(RC);
                // far values in flight stay valid across a general-path level:
                // a far edge either spans more than D + 1 levels or was folded
                // early by its wide level
                far_loads(st[(r + 1 + kD) % kNS], bd);
                long_store(sa, RC);
                records(st[(r + 1 + kD + kRF) % kNS], brf);
                __syncthreads();
                step++;
            }
        };
        while (step + kNS <= s1) unroll_seq(one, std::make_integer_sequence<int, kNS>{});
        for (; step < s1; step++) {
            pair_slow<S, FWD, false, BM, NXF>(kargs_here(), c.p0 / S, step, (LdsBytes *)c.win);
            __syncthreads();
        }
    }

    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (FWD) {
        if (c.lds_bins && NEAR)
            for (int i = lane; i < c.K * S; i += kLanes) {
                const int l = i / S, s = i % S;
                if (c.p0 + s < c.P) a.label_mem[(int64_t)(c.p0 + s) * c.K + l] = c.bins[i];
            }
        return;
    }
    if (!NEAR || a.seg_on) return;   // segmented: a separate pass takes the makespan
    // b: makespan M = max over v of tl + bl is reached at a node without
    // predecessors (tl = 0 there), i.e. at level 0; the path starts at the
    // smallest-id such node with bl == M (level 0 is sorted by id).
    const int32_t n0 = L > 0 ? c.pls[1].node_lo : 0;
#pragma unroll
    for (int s = 0; s < S; s++) {
        long long m = 0;
        for (int32_t i = lane; i < n0; i += kLanes) {
            const long long x = c.gval(c.vals[i].v[s]);
            m = x > m ? x : m;
        }
        m = wave_max_i64(m);
        int32_t first = INT32_MAX;
        for (int32_t i = lane; i < n0; i += kLanes)
            if (c.gval(c.vals[i].v[s]) == m) first = min(first, i);
#pragma unroll
        for (int off = kLanes / 2; off > 0; off >>= 1) first = min(first, __shfl_xor(first, off, kLanes));
        if (lane == 0 && c.p0 + s < c.P) {
            a.makespan[c.p0 + s] = m;
            if (a.start) a.start[c.p0 + s] = first == INT32_MAX ? -1 : first;
        }
    }
    (void)vmax;
}

template <int S, int BM, bool NXF>
__global__ __launch_bounds__(2 * kLanes) void k_sweep_pair(SweepArgs a) {
    extern __shared__ __align__(16) char smem[];
    if (a.gate != nullptr && *a.gate != a.gate_want) return;
    const int32_t n_slices = (a.P + S - 1) / S;
    const bool fwd = (int32_t)blockIdx.x >= n_slices;
    const int32_t slice = fwd ? blockIdx.x - n_slices : blockIdx.x;
    // both directions take BM (only the t chain keeps label sums)
    if (wave_id() == 0) {
        if (fwd)
            pair_chain<S, true, true, BM, false>(a, slice, smem);
        else
            pair_chain<S, false, true, BM, NXF>(a, slice, smem);
    } else {
        if (fwd)
            pair_chain<S, true, false, BM, false>(a, slice, smem);
        else
            pair_chain<S, false, false, BM, NXF>(a, slice, smem);
    }
}

// ---- wide levels of a single placement: grid-wide passes ----
// A level wider than the segmented chain's threshold is computed by the whole
// GPU between two chain launches: every in-edge (t) or out-edge (b) of the
// level is one task that folds its candidate into the owner's accumulator
// with a 64-bit atomic maximum (edge-parallel, so a hub costs no serial loop),
// then one task per node finalises it. All neighbours are final in the
// workspace. xt / xb: the t and b level (-1: none); acc_t / acc_b: one int64
// per node of the level, 0 on entry and reset to 0 on exit (the empty maximum).
__global__ void k_wide_edges(SweepArgs a, int32_t xt, int32_t xb, long long *acc_t,
                             long long *acc_b) {
    if (a.gate != nullptr && *a.gate != a.gate_want) return;
    using EL = Elem<true>;
    const int lb = a.lb, ob = a.ob;
    const int64_t t0 = xt >= 0 ? a.linfo[xt].in_e_lo : 0;
    const int64_t nt = xt >= 0 ? a.linfo[xt + 1].in_e_lo - t0 : 0;
    const int64_t b0 = xb >= 0 ? a.linfo[xb].out_e_lo : 0;
    const int64_t nb = xb >= 0 ? a.linfo[xb + 1].out_e_lo - b0 : 0;
    const int32_t tlo = xt >= 0 ? a.linfo[xt].node_lo : 0;
    const int32_t blo = xb >= 0 ? a.linfo[xb].node_lo : 0;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < nt + nb;
         i += (int64_t)gridDim.x * blockDim.x) {
        const bool fwd = i < nt;
        const EdgeRec16 r = fwd ? a.in_rec[t0 + i] : a.out_rec[b0 + (i - nt)];
        const int64_t g = fwd ? a.ftl[r.nb] : a.bll[r.nb];
        const int32_t own_lab = a.lab_w[r.own];
        const int64_t cand = EL::val(g, lb) + (EL::lab(g, lb) != own_lab ? r.cost : 0);
        (void)ob;
        if (fwd)
            atomicMax(&acc_t[r.own - tlo], (long long)cand);
        else
            atomicMax(&acc_b[r.own - blo], (long long)cand);
    }
}

__global__ void k_wide_nodes(SweepArgs a, int32_t xt, int32_t xb, long long *acc_t,
                             long long *acc_b) {
    if (a.gate != nullptr && *a.gate != a.gate_want) return;
    using EL = Elem<true>;
    const int lb = a.lb;
    const int32_t tlo = xt >= 0 ? a.linfo[xt].node_lo : 0;
    const int32_t nt = xt >= 0 ? a.linfo[xt + 1].node_lo - tlo : 0;
    const int32_t blo = xb >= 0 ? a.linfo[xb].node_lo : 0;
    const int32_t nb = xb >= 0 ? a.linfo[xb + 1].node_lo - blo : 0;
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < nt + nb;
         i += gridDim.x * blockDim.x) {
        const bool fwd = i < nt;
        const int32_t k = fwd ? i : i - nt;
        const int32_t v = (fwd ? tlo : blo) + k;
        long long *acc = fwd ? acc_t : acc_b;
        const int64_t m = acc[k];
        acc[k] = 0;
        const int64_t comp = a.node_rec[v].comp;
        const int64_t x = EL::make(m + comp, a.lab_w[v], lb);
        if (fwd)
            a.ftl[v] = x;
        else
            a.bll[v] = x;
    }
}

// makespan of a segmented single sweep: the largest bl over level 0
__global__ __launch_bounds__(256) void k_level0_makespan(SweepArgs a) {
    if (a.gate != nullptr && *a.gate != a.gate_want) return;
    using EL = Elem<true>;
    __shared__ long long s_m;
    if (threadIdx.x == 0) s_m = 0;
    __syncthreads();
    const int32_t n0 = a.L > 0 ? a.linfo[1].node_lo : 0;
    long long m = 0;
    for (int32_t v = threadIdx.x; v < n0; v += blockDim.x) {
        const long long x = EL::val(a.bll[v], a.lb);
        m = x > m ? x : m;
    }
    lds_max_i64(&s_m, m);
    __syncthreads();
    if (threadIdx.x == 0) *a.makespan = s_m;
}

// ---- structure: split each level's edges into span-1 and longer edges ----
__global__ void k_pair_flags(int64_t E, bool fwd, const int32_t *level, const int32_t *order,
                             const int32_t *nbr, const int32_t *own, int32_t *flag) {
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < E;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int32_t lv_nb = level[order[nbr[e]]], lv_ow = level[order[own[e]]];
        flag[e] = (fwd ? lv_ow - lv_nb : lv_nb - lv_ow) == 1 ? 1 : 0;
    }
}

__global__ void k_pair_levels(int32_t L, const int32_t *level_ptr, const int32_t *off,
                              const int32_t *near_rank, PairLevel *pl) {
    for (int32_t k = blockIdx.x * blockDim.x + threadIdx.x; k <= L + 1;
         k += gridDim.x * blockDim.x) {
        const int32_t lo = level_ptr[min(k, L)];
        const int32_t e = off[lo], e1 = off[level_ptr[min(k + 1, L)]];
        PairLevel x;
        x.node_lo = lo;
        x.near_lo = near_rank[e];
        x.far_lo = e - near_rank[e];
        // every far record, until the long-edge pass has put the ones that
        // read the workspace first and counted them (64 or fewer far records
        // are all task 0 in any order)
        x.n_gather = (e1 - near_rank[e1]) - x.far_lo;
        pl[k] = x;
    }
}

__global__ void k_pair_records(int64_t E, int32_t L, bool fwd, int32_t ob, const int32_t *level,
                               const int32_t *order, const int32_t *level_ptr, const int32_t *nbr,
                               const int32_t *own, const int64_t *cost, const int32_t *nb_orig,
                               const int32_t *near_rank, NearRec12 *nr, FarRec16 *fr) {
    const long long omax = (1ll << ob) - 1;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < E;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int32_t nb = nbr[e], ow = own[e];
        const int32_t lv_nb = level[order[nb]], lv_ow = level[order[ow]];
        const int32_t span = fwd ? lv_ow - lv_nb : lv_nb - lv_ow;
        const int32_t nb_lo = level_ptr[lv_nb];
        const uint32_t own_local = (uint32_t)(ow - level_ptr[lv_ow]) & 0xffffu;
        const uint32_t nb_local = (uint32_t)(nb - nb_lo);
        // the cost word (unsigned: when costs are too large for it, the
        // packed keys and these records go unused)
        const int64_t ck = fwd ? cost[e]
                               : (int64_t)(((uint64_t)cost[e] << ob) | (uint64_t)(omax - nb_orig[e]));
        if (span == 1) {
            NearRec12 r;
            r.ol = own_local | ((nb_local & 0xffffu) << 16);
            r.ck_lo = (uint32_t)ck;
            r.ck_hi = (uint32_t)((uint64_t)ck >> 32);
            nr[near_rank[e]] = r;
        } else {
            const int32_t w_nb = level_ptr[lv_nb + 1] - nb_lo;
            const int32_t step_nb = fwd ? lv_nb : L - 1 - lv_nb;
            const uint32_t rg = span > kD + 1 ? kNoRing
                                : w_nb <= kPNodes ? (uint32_t)((step_nb % kRS) * kPNodes) + nb_local
                                                  : kPreFolded;
            FarRec16 r;
            r.nb = nb;
            r.ol = own_local | (rg << 16);
            r.ck = ck;
            fr[e - near_rank[e]] = r;
        }
    }
}

// Long edges, one workgroup per block of kLongBlock steps: the block's far
// records whose neighbour finished by step kLongBlock * k - kLongLead (levels
// of the fast shape only: the others read the workspace), sorted by
// neighbour; distinct neighbours are listed in that order and the records
// pointed at their entry in the block's LDS buffer. A block with more than
// kLongCap distinct neighbours keeps the rest on the per-level gathers.
// Then each level's far records are reordered so that those still reading
// the workspace come first, and counted.
constexpr int kLongSort = 2048;   // >= kLongBlock * kNEf * kLanes
static_assert(kLongSort >= kLongBlock * kNEf * kLanes, "a block's far records fit the sort");

__device__ __forceinline__ bool fast_shape(const PairLevel &l0, const PairLevel &l1) {
    return l1.node_lo - l0.node_lo <= kPNodes && l1.near_lo - l0.near_lo <= kNEn * kLanes &&
           l1.far_lo - l0.far_lo <= kNEf * kLanes;
}

__device__ void long_assign(int32_t L, bool fwd, const PairLevel *pl, const int32_t *level,
                            const int32_t *order, FarRec16 *fr, int32_t *lsrc, int32_t k,
                            int32_t last, int32_t *key, int32_t *idx, int32_t *cnt_p) {
    int32_t &cnt = *cnt_p;
    if (threadIdx.x == 0) cnt = 0;
    __syncthreads();
    for (int32_t sx = k * kLongBlock; sx < min(L, (k + 1) * kLongBlock); sx++) {
        const int32_t x = fwd ? sx : L - 1 - sx;
        const PairLevel l0 = pl[x], l1 = pl[x + 1];
        if (!fast_shape(l0, l1)) continue;
        for (int32_t e = l0.far_lo + threadIdx.x; e < l1.far_lo; e += blockDim.x) {
            const FarRec16 r = fr[e];
            if ((r.ol >> 16) != kNoRing) continue;
            const int32_t lv = level[order[r.nb]];
            if ((fwd ? lv : L - 1 - lv) > last) continue;
            const int32_t p = atomicAdd(&cnt, 1);
            key[p] = r.nb;
            idx[p] = e;
        }
    }
    __syncthreads();
    const int32_t n = cnt;
    int32_t m = 1;
    while (m < n) m <<= 1;
    for (int32_t i = n + threadIdx.x; i < m; i += blockDim.x) {
        key[i] = INT32_MAX;
        idx[i] = -1;
    }
    __syncthreads();
    // bitonic sort by neighbour
    for (int32_t size = 2; size <= m; size <<= 1)
        for (int32_t stride = size >> 1; stride > 0; stride >>= 1) {
            for (int32_t i = threadIdx.x; i < m; i += blockDim.x) {
                const int32_t j = i ^ stride;
                if (j > i) {
                    const int32_t ki = key[i], kj = key[j];
                    if ((ki > kj) == ((i & size) == 0)) {
                        key[i] = kj;
                        key[j] = ki;
                        const int32_t t = idx[i];
                        idx[i] = idx[j];
                        idx[j] = t;
                    }
                }
            }
            __syncthreads();
        }
    if (threadIdx.x == 0) {
        int32_t slot = -1;
        for (int32_t i = 0; i < n; i++) {
            if (i == 0 || key[i] != key[i - 1]) {
                if (++slot == kLongCap) break;
                lsrc[(int64_t)k * kLongCap + slot] = key[i];
            }
            FarRec16 &r = fr[idx[i]];
            r.ol = (r.ol & 0xffffu) | ((kLongBase + (uint32_t)((k & 1) * kLongCap + slot)) << 16);
        }
    }
}

__global__ __launch_bounds__(256) void k_long_blocks(int32_t L, bool fwd, PairLevel *pl,
                                                      const int32_t *level, const int32_t *order,
                                                      FarRec16 *fr, int32_t *lsrc) {
    __shared__ int32_t key[kLongSort], idx[kLongSort];
    __shared__ int32_t cnt;
    __shared__ int wsum[256 / kLanes + 1];
    const int32_t k = blockIdx.x;
    const int32_t sx0 = k * kLongBlock, sx1 = min(L, sx0 + kLongBlock);
    const int32_t last = sx0 - kLongLead;   // latest neighbour step of a long edge
    if (last >= 0) long_assign(L, fwd, pl, level, order, fr, lsrc, k, last, key, idx, &cnt);
    __syncthreads();
    static_assert(kNEf * kLanes <= 256, "one far record per thread");
    for (int32_t sx = sx0; sx < sx1; sx++) {
        const int32_t x = fwd ? sx : L - 1 - sx;
        const PairLevel l0 = pl[x], l1 = pl[x + 1];
        if (!fast_shape(l0, l1)) continue;
        const int32_t nf = l1.far_lo - l0.far_lo;
        FarRec16 r{};
        int flag = 0;
        if ((int32_t)threadIdx.x < nf) {
            r = fr[l0.far_lo + threadIdx.x];
            flag = (r.ol >> 16) == kNoRing ? 1 : 0;
        }
        int total;
        const int before = block_excl_scan_i32(flag, wsum, &total);   // every read is done
        if ((int32_t)threadIdx.x < nf)
            fr[l0.far_lo + (flag ? before : total + (int32_t)threadIdx.x - before)] = r;
        if (threadIdx.x == 0) pl[x].n_gather = total;
        __syncthreads();
    }
}

// Edges a wide level folds early, in neighbour-grouped order (t: the CSR by
// source, b: the CSC by destination): span 2 .. D + 1, neighbour's level wider
// than the ring, owner's level narrow enough for the accumulators.
__global__ void k_pre_flags(int64_t E, bool fwd, const int32_t *level, const int32_t *order,
                            const int32_t *level_ptr, const int32_t *nbr, const int32_t *own,
                            int32_t *flag) {
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < E;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int32_t lv_nb = level[order[nbr[e]]], lv_ow = level[order[own[e]]];
        const int32_t span = fwd ? lv_ow - lv_nb : lv_nb - lv_ow;
        const int32_t w_nb = level_ptr[lv_nb + 1] - level_ptr[lv_nb];
        const int32_t w_ow = level_ptr[lv_ow + 1] - level_ptr[lv_ow];
        flag[e] = span >= 2 && span <= kD + 1 && w_nb > kPNodes && w_ow <= kPNodes ? 1 : 0;
    }
}

__global__ void k_pre_off(int32_t L, const int32_t *level_ptr, const int32_t *off,
                          const int32_t *rank, int32_t *preoff) {
    for (int32_t k = blockIdx.x * blockDim.x + threadIdx.x; k <= L; k += gridDim.x * blockDim.x)
        preoff[k] = rank[off[level_ptr[k]]];
}

__global__ void k_pre_records(int64_t E, bool fwd, int32_t ob, const int32_t *level,
                              const int32_t *order, const int32_t *level_ptr, const int32_t *nbr,
                              const int32_t *own, const int64_t *cost, const int32_t *rank,
                              PreRec16 *pre, int32_t *pretie) {
    const long long omax = (1ll << ob) - 1;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < E;
         e += (int64_t)gridDim.x * blockDim.x) {
        if (rank[e + 1] == rank[e]) continue;   // not flagged (rank: exclusive scan)
        const int32_t nb = nbr[e], ow = own[e];
        const int32_t lv_nb = level[order[nb]], lv_ow = level[order[ow]];
        const int32_t span = fwd ? lv_ow - lv_nb : lv_nb - lv_ow;
        PreRec16 r;
        r.nb = nb;
        r.os = (uint32_t)(ow - level_ptr[lv_ow]) | ((uint32_t)span << 16);
        r.cost = cost[e];
        pre[rank[e]] = r;
        if (!fwd) pretie[rank[e]] = (int32_t)(omax - order[nb]);
    }
}

}  // namespace

hipError_t launch_pre_flags(const Graph &g, bool fwd, int32_t *flag) {
    if (g.E == 0) return hipSuccess;
    const unsigned grid = (unsigned)std::min<int64_t>((g.E + 255) / 256, 65536);
    k_pre_flags<<<grid, 256, 0, g.stream>>>(g.E, fwd, g.level, g.order, g.level_ptr,
                                            fwd ? g.out_src : g.in_dst,
                                            fwd ? g.out_dst : g.in_src, flag);
    return hipGetLastError();
}

hipError_t launch_pre_split(const Graph &g, bool fwd, const int32_t *rank, int32_t *preoff,
                            PreRec16 *pre, int32_t *pretie) {
    k_pre_off<<<(unsigned)((g.L + 1 + 255) / 256), 256, 0, g.stream>>>(
        g.L, g.level_ptr, fwd ? g.out_off : g.in_off, rank, preoff);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || g.E == 0) return e;
    const unsigned grid = (unsigned)std::min<int64_t>((g.E + 255) / 256, 65536);
    k_pre_records<<<grid, 256, 0, g.stream>>>(
        g.E, fwd, succ_bits(g.V), g.level, g.order, g.level_ptr, fwd ? g.out_src : g.in_dst,
        fwd ? g.out_dst : g.in_src, fwd ? g.out_cost : g.in_cost, rank, pre, pretie);
    return hipGetLastError();
}

hipError_t launch_long_blocks(const Graph &g, bool fwd, PairLevel *pl, FarRec16 *fr,
                              int32_t *lsrc) {
    hipError_t e = launch_fill_i32(lsrc, long_list_elems(g.L), 0, g.stream);
    const int32_t n_blk = (g.L + kLongBlock - 1) / kLongBlock;
    if (e != hipSuccess || n_blk == 0 || g.E == 0) return e;
    k_long_blocks<<<(unsigned)n_blk, 256, 0, g.stream>>>(g.L, fwd, pl, g.level, g.order, fr, lsrc);
    return hipGetLastError();
}

hipError_t launch_pair_flags(const Graph &g, bool fwd, int32_t *flag) {
    if (g.E == 0) return hipSuccess;
    const unsigned grid = (unsigned)std::min<int64_t>((g.E + 255) / 256, 65536);
    k_pair_flags<<<grid, 256, 0, g.stream>>>(g.E, fwd, g.level, g.order,
                                             fwd ? g.in_src : g.out_dst,
                                             fwd ? g.in_dst : g.out_src, flag);
    return hipGetLastError();
}

hipError_t launch_pair_split(const Graph &g, bool fwd, const int32_t *near_rank, PairLevel *pl,
                             NearRec12 *nr, FarRec16 *fr) {
    k_pair_levels<<<(unsigned)((g.L + 2 + 255) / 256), 256, 0, g.stream>>>(
        g.L, g.level_ptr, fwd ? g.in_off : g.out_off, near_rank, pl);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || g.E == 0) return e;
    const unsigned grid = (unsigned)std::min<int64_t>((g.E + 255) / 256, 65536);
    k_pair_records<<<grid, 256, 0, g.stream>>>(
        g.E, g.L, fwd, succ_bits(g.V), g.level, g.order, g.level_ptr,
        fwd ? g.in_src : g.out_dst, fwd ? g.in_dst : g.out_src, fwd ? g.in_cost : g.out_cost,
        g.out_dst_orig, near_rank, nr, fr);
    return hipGetLastError();
}

template <int S>
hipError_t launch_pair(const SweepArgs &a, hipStream_t s) {
    const int32_t n_slices = (a.P + S - 1) / S;
    if (n_slices == 0) return hipSuccess;
    if (a.lb <= 0) return hipErrorInvalidValue;
    const size_t bins = a.K > 0 && a.K * S <= kPBinsCap ? (size_t)a.K * S * 8 : 0;
    const size_t lds = pair_lds_fixed<S>() + bins;
    // the batch reads 16-bit labels, and only it does
    if ((S == kBatchSlots) != (a.lab16 != 0)) return hipErrorInvalidValue;
    if (a.nxf) {   // links folded into the b values: batches only
        if constexpr (S == kBatchSlots) {
            if (a.K <= 0)
                k_sweep_pair<S, kBinsNone, true><<<2 * n_slices, 2 * kLanes, lds, s>>>(a);
            else if (bins > 0)
                k_sweep_pair<S, kBinsLds, true><<<2 * n_slices, 2 * kLanes, lds, s>>>(a);
            else
                k_sweep_pair<S, kBinsGlobal, true><<<2 * n_slices, 2 * kLanes, lds, s>>>(a);
        } else {
            return hipErrorInvalidValue;
        }
    } else if (a.K <= 0) {
        k_sweep_pair<S, kBinsNone, false><<<2 * n_slices, 2 * kLanes, lds, s>>>(a);
    } else if (bins > 0) {
        k_sweep_pair<S, kBinsLds, false><<<2 * n_slices, 2 * kLanes, lds, s>>>(a);
    } else {
        k_sweep_pair<S, kBinsGlobal, false><<<2 * n_slices, 2 * kLanes, lds, s>>>(a);
    }
    return hipGetLastError();
}

hipError_t launch_sweep_pair(const SweepArgs &a, hipStream_t s) {
    return launch_pair<kBatchSlots>(a, s);
}

hipError_t launch_wide_level(const SweepArgs &a, int32_t xt, int32_t xb, int64_t n_edges,
                             int32_t n_nodes, long long *acc_t, long long *acc_b, hipStream_t s) {
    if (a.lb <= 0 || a.P != 1) return hipErrorInvalidValue;
    const unsigned ge = (unsigned)std::max<int64_t>(1, std::min<int64_t>((n_edges + 255) / 256, 8192));
    k_wide_edges<<<ge, 256, 0, s>>>(a, xt, xb, acc_t, acc_b);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const unsigned gn = (unsigned)std::max<int64_t>(1, std::min<int64_t>((n_nodes + 255) / 256, 8192));
    k_wide_nodes<<<gn, 256, 0, s>>>(a, xt, xb, acc_t, acc_b);
    return hipGetLastError();
}

hipError_t launch_level0_makespan(const SweepArgs &a, hipStream_t s) {
    if (a.lb <= 0 || a.P != 1) return hipErrorInvalidValue;
    k_level0_makespan<<<1, 256, 0, s>>>(a);
    return hipGetLastError();
}

// One placement per chain: for a single placement (no label sums) the chain
// carries one value per node, which shortens its per-level step.
hipError_t launch_sweep_pair_one(const SweepArgs &a, hipStream_t s) {
    if (a.K > 0) return hipErrorInvalidValue;
    return launch_pair<1>(a, s);
}

}  // namespace pardnn
