// peel.hip -- the secondary clusters of graph slicing (paper Alg. 1 past its
// K primary paths, Sec. 3.1.1).
//
// Past K paths the weighted levels are no longer recomputed: every further
// path is found by walking the remaining graph with the priorities w = tl + bl
// of the last recomputation (the graph left after the K-th primary) until a
// dead end, and then leaves the graph with its edges. The walk starts at the
// remaining node without a remaining predecessor of largest w, steps to the
// remaining successor of largest w and stops at a node with no remaining
// successor; ties in w go to the smaller node id. New walks start until no
// node remains.
//
// Design for gfx950. The walk is one dependent chain over every remaining
// node, so it runs in ONE wave; everything that does not depend on the walk
// is prepared by data-parallel passes first:
//   * the remaining nodes are ranked by (w descending, id ascending) with a
//     stable radix sort, so "largest priority" becomes "smallest rank";
//   * the remaining edges are radix-sorted by (rank of source, rank of
//     destination): each node's successors come out in priority order, and
//     the best remaining successor is the first one not yet removed;
//   * one 32-byte record per rank holds the node's edge offset, out-degree and
//     its first six successors, so that a step of the walk usually needs a
//     single round trip to memory: it decrements the in-degrees of the current
//     node's successors (atomics with return) and loads the records of all of
//     them in the same go, before it knows which one comes next;
//   * the set of removed nodes and a three-level bitmap of the current
//     sources (remaining nodes whose remaining in-degree is zero) live in LDS
//     when they fit, so a priority test is one LDS read and the best source
//     one walk down the three levels;
//   * the sources a step creates are marked in the bitmap at the next step
//     (or when the walk ends, before the next start is chosen): the in-degree
//     atomics return later than the record loads, and this way their wait
//     overlaps the next step's loads (17 % off the walk).
// The walk writes ranks; a final data-parallel pass turns them into node ids
// and cluster numbers.
#include <algorithm>

#include "device_utils.h"
#include "internal.h"

namespace pardnn {

namespace {

constexpr int kBlock = 256;
constexpr int kInline = 6;   // successors held in a node's record

struct alignas(16) PeelRec {
    int32_t off, deg;
    int32_t s[kInline];
};
static_assert(sizeof(PeelRec) == 32, "a record is 8 words, one per lane of a group of 8");

inline unsigned grid_for(int64_t n, int block, int cap = 65536) {
    int64_t g = (n + block - 1) / block;
    if (g < 1) g = 1;
    if (g > cap) g = cap;
    return (unsigned)g;
}

inline size_t al256(size_t b) { return (b + 255) / 256 * 256; }

// words of the removed map and the three source levels for R ranks
struct MapDims {
    int32_t w0, w1, w2;
    __host__ __device__ explicit MapDims(int32_t R)
        : w0((R + 63) / 64), w1((w0 + 63) / 64), w2((w1 + 63) / 64) {}
    __host__ __device__ int32_t words() const { return 2 * w0 + w1 + w2; }
};

// Sort key of a node: bound - w for a remaining node (smaller = more urgent),
// bound + 1 for a removed one; values: the ids in ascending order.
__global__ void k_peel_keys(int32_t V, const int32_t *rank, const uint8_t *alive_lm,
                            const int64_t *tl, const int64_t *bl, uint64_t bound, uint64_t *key,
                            int32_t *ids) {
    for (int32_t v = blockIdx.x * blockDim.x + threadIdx.x; v < V; v += gridDim.x * blockDim.x) {
        const bool alive = alive_lm[rank[v]] != 0;
        key[v] = alive ? bound - (uint64_t)(tl[v] + bl[v]) : bound + 1;
        ids[v] = v;
    }
}

// prank[v] = priority rank of v (-1: not remaining); R = remaining nodes
__global__ void k_peel_rank(int32_t V, const uint64_t *key, uint64_t dead, const int32_t *sids,
                            int32_t *prank, int32_t *R) {
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < V; i += gridDim.x * blockDim.x) {
        const bool alive = key[i] != dead;
        prank[sids[i]] = alive ? i : -1;
        if (alive && (i + 1 == V || key[i + 1] == dead)) *R = i + 1;
    }
}

// remaining edges as (rank of source) * R + (rank of destination); the others
// sort last under `dead`; out- and in-degrees in rank space
__global__ void k_peel_edges(int64_t E, const int32_t *src, const int32_t *dst,
                             const int32_t *prank, const int32_t *Rp, uint64_t dead,
                             uint64_t *key, int32_t *val, int32_t *outdeg, int32_t *indeg) {
    const uint64_t R = (uint64_t)*Rp;
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < E;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int32_t a = prank[src[e]], b = prank[dst[e]];
        if (a >= 0 && b >= 0) {
            key[e] = (uint64_t)a * R + (uint64_t)b;
            val[e] = b;
            atomicAdd(&outdeg[a], 1);
            atomicAdd(&indeg[b], 1);
        } else {
            key[e] = dead;
            val[e] = -1;
        }
    }
}

__global__ void k_peel_records(int32_t V, const int32_t *Rp, const int32_t *off,
                               const int32_t *succ, PeelRec *rec) {
    const int32_t R = *Rp;
    for (int32_t r = blockIdx.x * blockDim.x + threadIdx.x; r < R && r < V;
         r += gridDim.x * blockDim.x) {
        PeelRec x;
        x.off = off[r];
        x.deg = off[r + 1] - x.off;
#pragma unroll
        for (int i = 0; i < kInline; i++) x.s[i] = i < x.deg ? succ[x.off + i] : -1;
        rec[r] = x;
    }
}

// the sources before the first walk: bit r of word i set when rank r = 64 i + b
// has no remaining predecessor
__global__ void k_peel_src_init(const int32_t *Rp, int32_t V, const int32_t *indeg,
                                uint64_t *s0) {
    const int32_t R = *Rp;
    const int32_t w0 = (R + 63) / 64;
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < w0 && i < (V + 63) / 64;
         i += gridDim.x * blockDim.x) {
        uint64_t x = 0;
        for (int b = 0; b < 64; b++) {
            const int32_t r = i * 64 + b;
            if (r < R && indeg[r] == 0) x |= 1ull << b;
        }
        s0[i] = x;
    }
}

// The primaries, already found, open the cluster list: cluster j < K holds
// path j; *p0 = the number of their nodes.
__global__ void k_peel_primaries(int32_t K, const int32_t *paths, int32_t stride,
                                 const int32_t *plen, int32_t *cl_off, int32_t *cl_nodes,
                                 int32_t *p0) {
    int32_t pos = 0;
    for (int32_t j = 0; j < K; j++) {
        const int32_t n = plen[j];
        if (threadIdx.x == 0) cl_off[j] = pos;
        for (int32_t i = threadIdx.x; i < n; i += blockDim.x)
            cl_nodes[pos + i] = paths[(int64_t)j * stride + i];
        pos += n;
    }
    if (threadIdx.x == 0) *p0 = pos;
}

// Bit maps through LDS (the usual case) or, for graphs too large for it,
// global memory at device scope; the walk is a single wave, and every access
// is an atomic or a device-coherent load, so its own writes are seen in order.
template <bool LDS>
struct Maps {
    uint64_t *rem, *s0, *s1, *s2;
    __device__ uint64_t ld(const uint64_t *p) const {
        if constexpr (LDS)
            return *p;
        else
            return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __device__ uint64_t or_(uint64_t *p, uint64_t m) const {
        return __hip_atomic_fetch_or(p, m, __ATOMIC_RELAXED,
                                     LDS ? __HIP_MEMORY_SCOPE_WORKGROUP : __HIP_MEMORY_SCOPE_AGENT);
    }
    __device__ uint64_t and_(uint64_t *p, uint64_t m) const {
        return __hip_atomic_fetch_and(p, m, __ATOMIC_RELAXED,
                                      LDS ? __HIP_MEMORY_SCOPE_WORKGROUP
                                          : __HIP_MEMORY_SCOPE_AGENT);
    }
    __device__ bool removed(int32_t r) const { return (ld(rem + (r >> 6)) >> (r & 63)) & 1ull; }
    __device__ void remove(int32_t r) const { or_(rem + (r >> 6), 1ull << (r & 63)); }
    __device__ void set_src(int32_t r) const {
        or_(s0 + (r >> 6), 1ull << (r & 63));
        or_(s1 + (r >> 12), 1ull << ((r >> 6) & 63));
        or_(s2 + (r >> 18), 1ull << ((r >> 12) & 63));
    }
    __device__ void clear_src(int32_t r) const {   // one lane
        const uint64_t b0 = 1ull << (r & 63), b1 = 1ull << ((r >> 6) & 63),
                       b2 = 1ull << ((r >> 12) & 63);
        if ((and_(s0 + (r >> 6), ~b0) & ~b0) != 0) return;
        if ((and_(s1 + (r >> 12), ~b1) & ~b1) != 0) return;
        and_(s2 + (r >> 18), ~b2);
    }
    // smallest source rank, -1 when there is none, -2 when a level names an
    // empty word below it (inconsistent maps; wave-uniform)
    __device__ int32_t first_src(int32_t w0, int32_t w1, int32_t w2) const {
        const int lane = lane_id();
        for (int32_t c = 0; c < w2; c += kWave) {
            const uint64_t x = c + lane < w2 ? ld(s2 + c + lane) : 0ull;
            const unsigned long long m = __ballot(x != 0ull);
            if (m == 0ull) continue;
            const int l = __ffsll((long long)m) - 1;
            const uint64_t x2 = __shfl(x, l, kWave);
            const int32_t i1 = (c + l) * 64 + (__ffsll((long long)x2) - 1);
            if (i1 >= w1) return -2;
            const uint64_t x1 = ld(s1 + i1);
            if (x1 == 0ull) return -2;
            const int32_t i0 = i1 * 64 + (__ffsll((long long)x1) - 1);
            if (i0 >= w0) return -2;
            const uint64_t x0 = ld(s0 + i0);
            if (x0 == 0ull) return -2;
            return i0 * 64 + (__ffsll((long long)x0) - 1);
        }
        return -1;
    }
};

// The walk, one wave. x holds field (lane & 7) of the current node's record.
// Lanes 2..7 carry its inline successors t; lanes 8 c .. 8 c + 7 load the
// record of successor c (c < 6) ahead of the choice. Steps past R (which a
// correct walk never takes) end the walk with err bit 1 set.
template <bool LDS>
__global__ __launch_bounds__(kWave) void k_peel_walk(const int32_t *Rp, int32_t K,
                                                     const PeelRec *rec, const int32_t *succ,
                                                     int32_t *indeg, const uint64_t *s0_init,
                                                     uint64_t *gmap, int32_t *cl_off,
                                                     int32_t *cl_nodes, const int32_t *p0,
                                                     int32_t *n_clusters, int32_t *err) {
    extern __shared__ __align__(16) uint64_t lmap[];
    const int lane = lane_id();
    const int32_t R = __builtin_amdgcn_readfirstlane(*Rp);
    const MapDims d(R);
    uint64_t *base = LDS ? lmap : gmap;
    Maps<LDS> mp{base, base + d.w0, base + 2 * d.w0, base + 2 * d.w0 + d.w1};
    const int32_t *recw = reinterpret_cast<const int32_t *>(rec);
    // maps: nothing removed; sources from the initial words, then levels 1, 2
    for (int32_t i = lane; i < d.w0; i += kWave) mp.rem[i] = 0;
    for (int32_t i = lane; i < d.w0; i += kWave) mp.s0[i] = s0_init[i];
    for (int32_t i = lane; i < d.w1 + d.w2; i += kWave) mp.s1[i] = 0;
    __builtin_amdgcn_s_waitcnt(0);
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
    for (int32_t i = lane; i < d.w0; i += kWave)
        if (mp.ld(mp.s0 + i) != 0ull) mp.or_(mp.s1 + (i >> 6), 1ull << (i & 63));
    __builtin_amdgcn_s_waitcnt(0);
    for (int32_t i = lane; i < d.w1; i += kWave)
        if (mp.ld(mp.s1 + i) != 0ull) mp.or_(mp.s2 + (i >> 6), 1ull << (i & 63));
    __builtin_amdgcn_s_waitcnt(0);

    int32_t pos = __builtin_amdgcn_readfirstlane(*p0);
    int32_t j = K, steps = 0;
    bool bad = false;
    while (!bad) {
        const int32_t s = mp.first_src(d.w0, d.w1, d.w2);
        if (s == -1) break;
        if (s < 0 || s >= R) {   // cannot happen for consistent maps
            bad = true;
            break;
        }
        if (lane == 0) {
            mp.clear_src(s);
            mp.remove(s);
            cl_off[j] = pos;
        }
        if constexpr (!LDS) __builtin_amdgcn_s_waitcnt(0);
        int32_t cur = s;
        int32_t x = recw[(int64_t)cur * 8 + (lane & 7)];
        // the source marks of a step are applied at the next one, so that
        // the wait for the in-degree atomics overlaps the next step's loads
        int32_t p_t = -1, p_old = 0, p_next = -1;
        bool p_rm = true;
        while (true) {
            if (++steps > R) {   // cannot happen for a correct walk
                bad = true;
                break;
            }
            if (lane == 0) cl_nodes[pos] = cur;
            pos++;
            const int32_t off = __builtin_amdgcn_readlane(x, 0);
            const int32_t deg = __builtin_amdgcn_readlane(x, 1);
            // inline successors in lanes 2..7, and the records of all of them
            const int32_t t = lane >= 2 && lane < 8 && lane - 2 < deg ? x : -1;
            const int c = lane >> 3;
            const int32_t tc = __shfl(x, 2 + (c < kInline ? c : 0), kWave);
            const bool load_c = c < kInline && c < deg && tc >= 0 && tc < R;
            const int32_t y = load_c ? recw[(int64_t)tc * 8 + (lane & 7)] : 0;
            const int32_t old = t >= 0 && t < R ? atomicSub(&indeg[t], 1) : 0;
            const bool rm = t >= 0 && t < R && mp.removed(t);
            if (p_t >= 0 && p_t < R && p_old == 1 && !p_rm && p_t != p_next) mp.set_src(p_t);
            int32_t next = -1;
            const unsigned long long m = __ballot(t >= 0 && t < R && !rm);
            if (m != 0ull) {
                const int fl = __ffsll((long long)m) - 1;
                next = __builtin_amdgcn_readlane(t, fl);
                x = __shfl(y, 8 * (fl - 2) + (lane & 7), kWave);
            }
            p_t = t;
            p_old = old;
            p_rm = rm;
            p_next = next;
            if (deg > kInline) {   // the rest of the list, 64 successors at a time
                bool need_rec = false;
                for (int32_t c0 = off + kInline; c0 < off + deg; c0 += kWave) {
                    const int32_t t2 = c0 + lane < off + deg ? succ[c0 + lane] : -1;
                    const bool ok = t2 >= 0 && t2 < R;
                    const int32_t old2 = ok ? atomicSub(&indeg[t2], 1) : 0;
                    const bool rm2 = ok && mp.removed(t2);
                    if (next < 0) {
                        const unsigned long long m2 = __ballot(ok && !rm2);
                        if (m2 != 0ull) {
                            next = __builtin_amdgcn_readlane(t2, __ffsll((long long)m2) - 1);
                            need_rec = true;
                        }
                    }
                    if (ok && old2 == 1 && !rm2 && t2 != next) mp.set_src(t2);
                }
                if (need_rec) x = recw[(int64_t)next * 8 + (lane & 7)];
            }
            if (next < 0) {
                if (p_t >= 0 && p_t < R && p_old == 1 && !p_rm && p_t != p_next) mp.set_src(p_t);
                break;
            }
            if (lane == 0) mp.remove(next);
            if constexpr (!LDS) __builtin_amdgcn_s_waitcnt(0);
            cur = next;
        }
        j++;
    }
    if (lane == 0) {
        cl_off[j] = pos;
        *n_clusters = j;
        if (bad) atomicOr(err, 1);
    }
}

// ranks -> node ids, and each node's cluster (the last cl_off[j] <= pos)
__global__ void k_peel_finish(int32_t V, const int32_t *p0, const int32_t *n_clusters, int32_t K,
                              const int32_t *cl_off, const int32_t *sids, int32_t *cl_nodes,
                              int32_t *cluster) {
    const int32_t start = *p0, n = *n_clusters;
    for (int32_t pos = start + blockIdx.x * blockDim.x + threadIdx.x; pos < V;
         pos += gridDim.x * blockDim.x) {
        const int32_t r = cl_nodes[pos];
        if ((uint32_t)r >= (uint32_t)V) {   // not written: the walk stopped early
            cl_nodes[pos] = -1;
            continue;
        }
        const int32_t o = sids[r];
        cl_nodes[pos] = o;
        int32_t lo = K, hi = n - 1;   // cl_off[lo] <= pos < cl_off[hi + 1]
        while (lo < hi) {
            const int32_t mid = (lo + hi + 1) >> 1;
            if (cl_off[mid] <= pos)
                lo = mid;
            else
                hi = mid - 1;
        }
        cluster[o] = lo;
    }
}

struct PeelLayout {
    size_t key, key_s, ids, sids, prank, scal, ekey, ekey_s, eval, succ, outdeg, indeg, off, ws,
        rec, s0, gmap, temp, total;
    PeelLayout(int32_t V, int64_t E) {
        size_t o = 0;
        auto take = [&](size_t bytes) {
            const size_t at = o;
            o += al256(bytes);
            return at;
        };
        const size_t v = (size_t)std::max(V, 1), e = (size_t)std::max<int64_t>(E, 1);
        key = take(v * 8);
        key_s = take(v * 8);
        ids = take(v * 4);
        sids = take(v * 4);
        prank = take(v * 4);
        scal = take(16);   // R, p0
        ekey = take(e * 8);
        ekey_s = take(e * 8);
        eval = take(e * 4);
        succ = take(e * 4);
        outdeg = take((v + 1) * 4);
        indeg = take(v * 4);
        off = take((v + 1) * 4);
        ws = take(scan_workspace_elems((int32_t)v) * 4);
        rec = take(v * sizeof(PeelRec));
        s0 = take((size_t)MapDims((int32_t)v).w0 * 8);
        gmap = take((size_t)MapDims((int32_t)v).words() * 8);
        temp = take(std::max(sort_pairs_scratch_bytes((int32_t)v, 8),
                             sort_pairs_scratch_bytes((int32_t)e, 8)));
        total = o;
    }
};

template <class T>
T *at_off(void *base, size_t off) {
    return reinterpret_cast<T *>(reinterpret_cast<char *>(base) + off);
}

}  // namespace

size_t peel_scratch_bytes(int32_t V, int64_t E) { return PeelLayout(V, E).total; }

size_t peel_lds_bytes(int32_t V) { return (size_t)MapDims(V).words() * 8; }

hipError_t launch_slice_secondaries(const Graph &g, int32_t K, const int32_t *paths,
                                    int32_t stride, const int32_t *plen, const int64_t *tl,
                                    const int64_t *bl, const uint8_t *alive_lm, int32_t *cluster,
                                    int32_t *cl_off, int32_t *cl_nodes, int32_t *n_clusters,
                                    void *scratch, bool lds_maps, int32_t *err) {
    const int32_t V = g.V;
    const int64_t E = g.E;
    const PeelLayout L(V, E);
    hipStream_t s = g.stream;
    uint64_t *key = at_off<uint64_t>(scratch, L.key), *key_s = at_off<uint64_t>(scratch, L.key_s);
    int32_t *ids = at_off<int32_t>(scratch, L.ids), *sids = at_off<int32_t>(scratch, L.sids);
    int32_t *prank = at_off<int32_t>(scratch, L.prank);
    int32_t *Rp = at_off<int32_t>(scratch, L.scal), *p0 = Rp + 1;
    uint64_t *ekey = at_off<uint64_t>(scratch, L.ekey);
    uint64_t *ekey_s = at_off<uint64_t>(scratch, L.ekey_s);
    int32_t *eval = at_off<int32_t>(scratch, L.eval), *succ = at_off<int32_t>(scratch, L.succ);
    int32_t *outdeg = at_off<int32_t>(scratch, L.outdeg);
    int32_t *indeg = at_off<int32_t>(scratch, L.indeg), *off = at_off<int32_t>(scratch, L.off);
    int32_t *ws = at_off<int32_t>(scratch, L.ws);
    PeelRec *rec = at_off<PeelRec>(scratch, L.rec);
    uint64_t *s0 = at_off<uint64_t>(scratch, L.s0), *gmap = at_off<uint64_t>(scratch, L.gmap);
    void *temp = at_off<char>(scratch, L.temp);
    hipError_t e;
    k_peel_primaries<<<1, kBlock, 0, s>>>(K, paths, stride, plen, cl_off, cl_nodes, p0);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = launch_fill_i32(Rp, 1, 0, s)) != hipSuccess) return e;
    if (V > 0) {
        const uint64_t bound = (uint64_t)g.weight_bound;
        int bits = 1;
        while (bits < 64 && ((bound + 1) >> bits) != 0) bits++;
        k_peel_keys<<<grid_for(V, kBlock), kBlock, 0, s>>>(V, g.rank, alive_lm, tl, bl, bound,
                                                           key, ids);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if ((e = sort_pairs_u64(key, key_s, ids, sids, V, 0, bits, temp, s)) != hipSuccess)
            return e;
        k_peel_rank<<<grid_for(V, kBlock), kBlock, 0, s>>>(V, key_s, bound + 1, sids, prank, Rp);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if ((e = launch_fill_i32(outdeg, (int64_t)V + 1, 0, s)) != hipSuccess) return e;
        if ((e = launch_fill_i32(indeg, V, 0, s)) != hipSuccess) return e;
        if (E > 0) {
            const uint64_t dead = (uint64_t)V * (uint64_t)V;   // above every live key
            int ebits = 1;
            while (ebits < 64 && (dead >> ebits) != 0) ebits++;
            k_peel_edges<<<grid_for(E, kBlock), kBlock, 0, s>>>(E, g.e_src, g.e_dst, prank, Rp,
                                                                dead, ekey, eval, outdeg, indeg);
            if ((e = hipGetLastError()) != hipSuccess) return e;
            if ((e = sort_pairs_u64(ekey, ekey_s, eval, succ, (int32_t)E, 0, ebits, temp, s)) !=
                hipSuccess)
                return e;
        }
        if ((e = launch_exclusive_scan(outdeg, off, V, ws, s)) != hipSuccess) return e;
        k_peel_records<<<grid_for(V, kBlock), kBlock, 0, s>>>(V, Rp, off, succ, rec);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        k_peel_src_init<<<grid_for((V + 63) / 64, kBlock), kBlock, 0, s>>>(Rp, V, indeg, s0);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (lds_maps) {
        k_peel_walk<true><<<1, kWave, peel_lds_bytes(V), s>>>(
            Rp, K, rec, succ, indeg, s0, gmap, cl_off, cl_nodes, p0, n_clusters, err);
    } else {
        k_peel_walk<false><<<1, kWave, 0, s>>>(Rp, K, rec, succ, indeg, s0, gmap, cl_off,
                                               cl_nodes, p0, n_clusters, err);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (V == 0) return hipSuccess;
    k_peel_finish<<<grid_for(V, kBlock), kBlock, 0, s>>>(V, p0, n_clusters, K, cl_off, sids,
                                                         cl_nodes, cluster);
    return hipGetLastError();
}

}  // namespace pardnn
