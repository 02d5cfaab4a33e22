// labelmem.hip -- memory per device label and placement updates.
//
// Memory Heuristic II (paper Sec. 3.2) balances per-partition memory totals;
// without its residual/normal split these totals are
//   label_mem[k] = sum of mem(v) over nodes v placed on label k,
// compared against the device capacity, of which the paper keeps 90 % (Sec. 4):
//   overflow[k] = max(0, label_mem[k] - capacity[k]).
// Node moves between partitions (Sec. 3.2) update the placement.
//
// Design for gfx950: the label sum is a segmented reduction into a handful of
// bins, so each workgroup privatises the bins in LDS (ds_add_u64) and flushes
// them with one global 64-bit atomic per bin. Building a batch of successive
// placements marks each (node, step) with its last move index (atomicMax keeps
// the latest move deterministic) and then forward-fills every placement-minor
// row with one wave, a 64-lane max-scan per chunk of steps.
#include <type_traits>


#include "device_utils.h"
#include "internal.h"

namespace pardnn {

namespace {

constexpr int kBlock = 256;
constexpr int kLdsBins = 4096;

// S labels of one node in a slice, stored with one access
template <int S>
struct alignas(4 * S) LabPack {
    int32_t v[S];
    // the same bytes as one scalar or vector word, for non-temporal stores
    using Word = typename std::conditional<
        S == 1, int32_t,
        typename std::conditional<S == 2, long long,
                                  int __attribute__((ext_vector_type(4)))>::type>::type;
    static_assert(S == 1 || S == 2 || S == 4, "one, two or four slots per slice");
};

// two labels as 16-bit halves of one word (the 16-bit label layout; the
// labels were checked against the full values)
__device__ __forceinline__ uint32_t pack16x2(int32_t a, int32_t b) {
    return (uint32_t)(uint16_t)a | ((uint32_t)(uint16_t)b << 16);
}

inline unsigned grid_for(int64_t n, int block, int cap = 65536) {
    int64_t g = (n + block - 1) / block;
    if (g < 1) g = 1;
    if (g > cap) g = cap;
    return (unsigned)g;
}

__global__ __launch_bounds__(kBlock) void k_label_sum(int32_t V, const int32_t *placement,
                                                      const int64_t *mem, int32_t K,
                                                      int64_t *label_mem, int32_t *err) {
    __shared__ long long bins[kLdsBins];
    const bool lds = K <= kLdsBins;
    if (lds) {
        for (int i = threadIdx.x; i < K; i += kBlock) bins[i] = 0;
        __syncthreads();
    }
    bool bad = false;
    for (int32_t v = blockIdx.x * kBlock + threadIdx.x; v < V; v += gridDim.x * kBlock) {
        const int32_t l = placement[v];
        if (l < 0 || l >= K) {
            bad = true;
            continue;
        }
        if (lds)
            lds_add_i64(&bins[l], mem[v]);
        else
            atomicAdd((unsigned long long *)&label_mem[l], (unsigned long long)mem[v]);
    }
    if (bad) atomicOr(err, 1);
    if (lds) {
        __syncthreads();
        for (int i = threadIdx.x; i < K; i += kBlock)
            if (bins[i] != 0)
                atomicAdd((unsigned long long *)&label_mem[i], (unsigned long long)bins[i]);
    }
}

// overflow[i] = max(0, label_mem[i] - capacity[i % K]) over n entries; flags
// negative capacities. Either output or capacity may be null.
__global__ void k_overflow(int64_t n, int32_t K, const int64_t *capacity,
                           const int64_t *label_mem, int64_t *overflow, int32_t *err) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        if (capacity == nullptr) {
            if (overflow) overflow[i] = 0;
            continue;
        }
        const int64_t cap = capacity[i % K];
        if (cap < 0) {
            atomicOr(err, 2);
            if (overflow) overflow[i] = 0;
            continue;
        }
        const int64_t s = label_mem[i];
        if (overflow) overflow[i] = s > cap ? s - cap : 0;
    }
}

__global__ void k_moves_mark(int32_t n, const int32_t *node, int32_t V, int32_t *stamp,
                             int32_t *err) {
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
        const int32_t v = node[i];
        if (v < 0 || v >= V)
            atomicOr(err, 1);
        else
            atomicMax(&stamp[v], i);
    }
}

__global__ void k_moves_apply(int32_t n, const int32_t *node, const int32_t *label, int32_t V,
                              int32_t *stamp, int32_t *placement, const int32_t *err) {
    const bool ok = *err == 0;
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
        const int32_t v = node[i];
        if (v < 0 || v >= V) continue;
        if (ok && stamp[v] == i) placement[v] = label[i];
    }
}

__global__ void k_moves_reset(int32_t n, const int32_t *node, int32_t V, int32_t *stamp) {
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
        const int32_t v = node[i];
        if (v >= 0 && v < V) stamp[v] = -1;
    }
}

// Mark (node, step) with the index of the last move of that node in that step.
__global__ void k_bp_mark(int64_t M, int32_t P, const int64_t *step_ptr, const int32_t *node,
                          int32_t V, int32_t *mat, int32_t *err) {
    for (int64_t m = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; m < M;
         m += (int64_t)gridDim.x * blockDim.x) {
        // step of move m: largest p with step_ptr[p] <= m
        int32_t lo = 0, hi = P;
        while (hi - lo > 1) {
            int32_t mid = (lo + hi) >> 1;
            if (step_ptr[mid] <= m)
                lo = mid;
            else
                hi = mid;
        }
        const int32_t v = node[m];
        if (v < 0 || v >= V) {
            atomicOr(err, 1);
            continue;
        }
        atomicMax(&mat[(int64_t)v * P + lo], (int32_t)m);
    }
}

// One wave per node row: value(p) = label of the latest move at a step <= p,
// else base. Moves within a row are in step order, so a running "last marked
// step" (inclusive max-scan over lanes) selects the move.
__global__ void k_bp_fill(int32_t V, int32_t P, const int32_t *base, const int32_t *label,
                          int32_t *mat) {
    const int lane = lane_id();
    const int64_t waves = (int64_t)gridDim.x * (blockDim.x / kWave);
    for (int64_t v = (int64_t)blockIdx.x * (blockDim.x / kWave) + wave_id(); v < V; v += waves) {
        int32_t carry = base[v];
        int32_t *row = mat + v * P;
        for (int32_t c0 = 0; c0 < P; c0 += kWave) {
            const int32_t p = c0 + lane;
            const int32_t m = p < P ? row[p] : -1;
            int32_t last = m >= 0 ? lane : -1;
#pragma unroll
            for (int off = 1; off < kWave; off <<= 1) {
                int32_t y = __shfl_up(last, off, kWave);
                if (lane >= off) last = max(last, y);
            }
            const int32_t mm = __shfl(m, last < 0 ? 0 : last, kWave);
            const int32_t val = last >= 0 ? label[mm] : carry;
            if (p < P) row[p] = val;
            carry = __shfl(val, kWave - 1, kWave);
        }
    }
}

// Moves grouped by node: one stable radix sort of the node ids over the move
// indices, so that each node's moves lie together in move order, with no
// per-node atomics and no counting pass. An id outside [0, V) is flagged and sorted
// past every node as V. Each node's range comes from a binary search of the
// sorted ids; the entries {step, move index, label} are gathered in sorted
// order.
__global__ void k_mv_keys(int64_t M, const int32_t *node, int32_t V, uint32_t *key, int32_t *idx,
                          int32_t *err) {
    for (int64_t m = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; m < M;
         m += (int64_t)gridDim.x * blockDim.x) {
        const int32_t v = node[m];
        const bool bad = v < 0 || v >= V;
        if (bad) atomicOr(err, 1);
        key[m] = bad ? (uint32_t)V : (uint32_t)v;
        idx[m] = (int32_t)m;
    }
}

// off[v] = first sorted position with id >= v, for v in [0, V]
__global__ void k_mv_off(int32_t V, int64_t M, const uint32_t *key, int32_t *off) {
    for (int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; v <= V;
         v += (int64_t)gridDim.x * blockDim.x) {
        int64_t lo = 0, hi = M;   // answer in [lo, hi]
        while (lo < hi) {
            const int64_t mid = (lo + hi) >> 1;
            if (key[mid] < (uint32_t)v)
                lo = mid + 1;
            else
                hi = mid;
        }
        off[v] = (int32_t)lo;
    }
}

__global__ void k_mv_gather(int64_t M, int32_t P, const int64_t *step_ptr, const uint32_t *key,
                            const int32_t *idx, const int32_t *label, int32_t V, int4 *ent) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < M;
         i += (int64_t)gridDim.x * blockDim.x) {
        if (key[i] >= (uint32_t)V) continue;
        const int32_t m = idx[i];
        // step of move m: largest p with step_ptr[p] <= m
        int32_t lo = 0, hi = P;
        while (hi - lo > 1) {
            const int32_t mid = (lo + hi) >> 1;
            if (step_ptr[mid] <= m)
                lo = mid;
            else
                hi = mid;
        }
        ent[i] = make_int4(lo, m, label[m], 0);
    }
}

// Labels of successive placements straight into the sweep's slice-major
// workspace lab_w[slice][v][s] (v level-major, placement p = slice * S + s).
// A workgroup owns 64 consecutive level-major nodes; each wave keeps the move
// lists of its 16 node rows in registers (entry `lane` of a list of at most
// 64 moves; longer lists are re-read per chunk). For a chunk of 64 placements
// a row's value at lane p is the label of its latest move with a step in
// [c0, c0 + p], else the row's label before the chunk: the moves that fall in
// the chunk (a ballot, usually none or one) are broadcast one at a time. The
// rows go through an LDS tile that is written out slice by slice as
// contiguous runs.
template <int S>
__global__ __launch_bounds__(256) void k_moves_to_slices(int32_t V, int32_t P,
                                                         const int32_t *order,
                                                         const int32_t *base,
                                                         const int32_t *mv_off,
                                                         const int4 *mv_ent, int32_t *lab_w,
                                                         int64_t lab_stride, int32_t K,
                                                         int32_t *err, int32_t *fit,
                                                         uint32_t fit_limit, int lab16,
                                                         const int32_t *gate, int32_t gate_want) {
    if (gate != nullptr && *gate != gate_want) return;   // (uniform)
    constexpr int TV = 64, TP = 64, NW = 256 / kWave, RW = TV / NW;
    __shared__ int32_t tile[TV][TP + 1];
    const int lane = lane_id(), w = wave_id();
    const int32_t v0 = blockIdx.x * TV;
    const int32_t n_slices = (P + S - 1) / S;
    int32_t lo[RW], cnt[RW], carry[RW];
    int4 ent[RW];
#pragma unroll
    for (int j = 0; j < RW; j++) {
        const int32_t v = v0 + w + j * NW;
        const int32_t o = v < V ? order[v] : -1;
        lo[j] = o >= 0 ? mv_off[o] : 0;
        cnt[j] = o >= 0 ? mv_off[o + 1] - lo[j] : 0;
        carry[j] = o >= 0 ? base[o] : 0;
    }
#pragma unroll
    for (int j = 0; j < RW; j++)
        ent[j] = lane < cnt[j] ? mv_ent[lo[j] + lane] : make_int4(-1, -1, 0, 0);
    // the largest label (as unsigned: a negative one counts as huge) over
    // this lane's columns, checked against K and fit_limit once at the end
    // instead of at every store. Columns past the last placement repeat its
    // labels (every move applies there) and rows past the last node hold 0,
    // so neither needs a mask.
    uint32_t umax = 0;
    // fold move x (uniform) into lane's value if it applies at lane's placement
    auto apply = [&](int32_t c0, int32_t st, int32_t m, int32_t lab, int32_t &best,
                     int32_t &val) {
        if (st - c0 <= lane && m > best) {
            best = m;
            val = lab;
        }
    };
    for (int32_t c0 = 0; c0 < n_slices * S; c0 += TP) {
#pragma unroll
        for (int j = 0; j < RW; j++) {
            int32_t val = carry[j], best = -1;
            if (cnt[j] <= kWave) {
                unsigned long long mask = __ballot(ent[j].x >= c0 && ent[j].x < c0 + TP);
                while (mask) {
                    const int e = __builtin_ctzll(mask);
                    mask &= mask - 1;
                    apply(c0, __builtin_amdgcn_readlane(ent[j].x, e),
                          __builtin_amdgcn_readlane(ent[j].y, e),
                          __builtin_amdgcn_readlane(ent[j].z, e), best, val);
                }
            } else {
                for (int32_t g = 0; g < cnt[j]; g += kWave) {
                    const int4 x = g + lane < cnt[j] ? mv_ent[lo[j] + g + lane]
                                                     : make_int4(-1, -1, 0, 0);
                    unsigned long long mask = __ballot(x.x >= c0 && x.x < c0 + TP);
                    while (mask) {
                        const int e = __builtin_ctzll(mask);
                        mask &= mask - 1;
                        apply(c0, __builtin_amdgcn_readlane(x.x, e),
                              __builtin_amdgcn_readlane(x.y, e),
                              __builtin_amdgcn_readlane(x.z, e), best, val);
                    }
                }
            }
            tile[w + j * NW][lane] = val;
            carry[j] = __builtin_amdgcn_readlane(val, kWave - 1);
            umax = max(umax, (uint32_t)val);
        }
        __syncthreads();
        const int32_t sl0 = c0 / S;
        const int n_sl = min(TP / S, n_slices - sl0);
        // streamed: the sweep reads these long after, and dirty lines left in
        // L2 would be written back during the sweep. Two adjacent nodes of
        // one slice per thread (one 16-byte store for two slots per slice).
        constexpr int NP = S == 2 ? 2 : 1;
        using W = typename LabPack<S * NP>::Word;
        for (int i = threadIdx.x; i < n_sl * (TV / NP); i += 256) {
            const int sl = i / (TV / NP), r = NP * (i % (TV / NP));
            const int32_t v = v0 + r;
            if (v >= V) continue;
            if constexpr (S == 2) {
                if (lab16) {   // 16-bit labels: 8 bytes for two nodes
                    uint32_t *d16 = reinterpret_cast<uint32_t *>(
                        reinterpret_cast<uint16_t *>(lab_w) + (int64_t)(sl0 + sl) * lab_stride +
                        (int64_t)v * 2);
                    const uint32_t w0 = pack16x2(tile[r][sl * 2], tile[r][sl * 2 + 1]);
                    if (v + 1 < V) {
                        typedef uint32_t u2 __attribute__((ext_vector_type(2)));
                        const u2 x = {w0, pack16x2(tile[r + 1][sl * 2], tile[r + 1][sl * 2 + 1])};
                        __builtin_nontemporal_store(x, reinterpret_cast<u2 *>(d16));
                    } else {
                        __builtin_nontemporal_store(w0, d16);
                    }
                    continue;
                }
            }
            int32_t *dst = lab_w + (int64_t)(sl0 + sl) * lab_stride + (int64_t)v * S;
            if (NP == 1 || v + 1 < V) {
                LabPack<S * NP> x;
#pragma unroll
                for (int q = 0; q < S * NP; q++) x.v[q] = tile[r + q / S][sl * S + q % S];
                __builtin_nontemporal_store(*reinterpret_cast<const W *>(&x),
                                            reinterpret_cast<W *>(dst));
            } else {   // the graph's last node alone
                LabPack<S> x;
#pragma unroll
                for (int q = 0; q < S; q++) x.v[q] = tile[r][sl * S + q];
                using W1 = typename LabPack<S>::Word;
                __builtin_nontemporal_store(*reinterpret_cast<const W1 *>(&x),
                                            reinterpret_cast<W1 *>(dst));
            }
        }
        __syncthreads();
    }
    if (K > 0 && umax >= (uint32_t)K) atomicOr(err, 1);
    if (fit != nullptr && umax >= fit_limit) *fit = 0;
}

// The same labels with one lane per level-major node, for schedules with a
// few moves per node. The workgroup first stages the move lists of its 256
// nodes, {step, label} in move order, in LDS (a workgroup whose lists hold
// more than kLaneMoves entries reads them from global memory instead); then
// each lane walks the slices in order, keeping its node's current label and
// next move, takes every move whose step is at most the placement, and writes
// the slice's S labels with one store. Consecutive lanes hold consecutive
// nodes, so each wave's store is one contiguous run of 64 x 4S bytes, and the
// only memory operations in the walk are these stores (the move reads come
// from LDS), so no wait on the stores is ever needed.
constexpr int kLaneMoves = 3584;   // LDS entries per workgroup (28 KB)
constexpr int kLaneMovesPerNode = 11;   // the host takes this kernel up to M <= 11 V

template <int S>
__global__ __launch_bounds__(256) void k_moves_lanes(int32_t V, int32_t P, const int32_t *order,
                                                     const int32_t *base, const int32_t *mv_off,
                                                     const int4 *mv_ent, int32_t *lab_w,
                                                     int64_t lab_stride, int32_t K, int32_t *err,
                                                     int32_t *fit, uint32_t fit_limit, int lab16,
                                                     const int32_t *gate, int32_t gate_want) {
    if (gate != nullptr && *gate != gate_want) return;   // (uniform)
    __shared__ int2 mv[kLaneMoves];
    __shared__ int wsum[256 / kWave + 1];
    const int32_t v = blockIdx.x * 256 + threadIdx.x;
    const int32_t o = v < V ? order[v] : -1;
    const int32_t lo = o >= 0 ? mv_off[o] : 0;
    const int32_t cnt = o >= 0 ? mv_off[o + 1] - lo : 0;
    const int32_t lab0 = o >= 0 ? base[o] : 0;
    int total;
    const int32_t at = block_excl_scan_i32(cnt, wsum, &total);
    const bool in_lds = total <= kLaneMoves;   // uniform over the workgroup
    if (in_lds) {
        for (int32_t k = 0; k < cnt; k += 4) {   // four loads in flight per lane
            int4 e[4];
#pragma unroll
            for (int j = 0; j < 4; j++)
                if (k + j < cnt) e[j] = mv_ent[lo + k + j];
#pragma unroll
            for (int j = 0; j < 4; j++)
                if (k + j < cnt) mv[at + k + j] = make_int2(e[j].x, e[j].z);
        }
    }
    __syncthreads();
    const int32_t n_slices = (P + S - 1) / S;
    uint32_t umax = 0;
    // the walk, with move k of the lane's list read by get(k)
    auto walk = [&](auto get) {
        constexpr int32_t kNone = INT32_MAX;   // past the last move
        int32_t cur = lab0, k = 0;
        int2 nx = cnt > 0 ? get(0) : make_int2(kNone, 0);
        // 32-bit labels at dst, or (16-bit layout, S = 2) one word per node
        int32_t *dst = lab_w + (int64_t)min(v, V - 1) * S;
        uint32_t *d16 = reinterpret_cast<uint32_t *>(reinterpret_cast<uint16_t *>(lab_w) +
                                                     (int64_t)min(v, V - 1) * 2);
        const int64_t step16 = lab_stride / 2;   // words per slice (the stride is even)
        for (int32_t sl = 0; sl < n_slices; sl++, dst += lab_stride, d16 += step16) {
            LabPack<S> x;
#pragma unroll
            for (int q = 0; q < S; q++) {
                const int32_t p = sl * S + q;   // past P every move applies
                while (nx.x <= p) {
                    cur = nx.y;
                    k++;
                    nx = k < cnt ? get(k) : make_int2(kNone, 0);
                }
                x.v[q] = cur;
                umax = max(umax, (uint32_t)cur);
            }
            if (v < V) {
                if constexpr (S == 2) {
                    if (lab16) {
                        __builtin_nontemporal_store(pack16x2(x.v[0], x.v[1]), d16);
                        continue;
                    }
                }
                __builtin_nontemporal_store(*reinterpret_cast<const typename LabPack<S>::Word *>(&x),
                                            reinterpret_cast<typename LabPack<S>::Word *>(dst));
            }
        }
    };
    if (in_lds)
        walk([&](int32_t k) { return mv[at + k]; });
    else
        walk([&](int32_t k) {
            const int4 e = mv_ent[lo + k];
            return make_int2(e.x, e.z);
        });
    if (K > 0 && umax >= (uint32_t)K) atomicOr(err, 1);
    if (fit != nullptr && umax >= fit_limit) *fit = 0;
}

}  // namespace

namespace {

// sorted id bits: ids run over [0, V] (V marks an invalid id)
unsigned mv_key_bits(int32_t V) {
    unsigned bits = 1;
    while (bits < 32 && ((uint32_t)V >> bits) != 0) bits++;
    return bits;
}

size_t mv_sort_temp_bytes(int32_t, int64_t M) { return sort_pairs_scratch_bytes((int32_t)M, 4); }

constexpr size_t al64(size_t n) { return (n + 63) / 64 * 64; }   // int32 elements, 256 B

}  // namespace

size_t moves_scratch_elems(int32_t V, int64_t M) {
    // off [V + 1], ids and move indices before and after the sort [M] each,
    // the entries (int4) [M], the sort's temporary storage; 256-byte aligned
    return al64((size_t)V + 1) + 4 * al64((size_t)M) + 4 * al64((size_t)M) +
           al64((mv_sort_temp_bytes(V, M) + 3) / 4);
}

namespace {

// the grouped moves in the scratch (see moves_scratch_elems)
struct MovesScratch {
    int32_t *off;
    uint32_t *key_in, *key_out;
    int32_t *idx_in, *idx_out;
    int4 *ent;
    void *temp;
};
MovesScratch moves_scratch(int32_t V, int64_t M, int32_t *scratch) {
    const size_t m64 = al64((size_t)M);
    MovesScratch m;
    m.off = scratch;
    m.key_in = reinterpret_cast<uint32_t *>(m.off + al64((size_t)V + 1));
    m.key_out = m.key_in + m64;
    m.idx_in = reinterpret_cast<int32_t *>(m.key_out + m64);
    m.idx_out = m.idx_in + m64;
    m.ent = reinterpret_cast<int4 *>(m.idx_out + m64);
    m.temp = reinterpret_cast<int32_t *>(m.ent) + 4 * m64;
    return m;
}

// the labels of every slice from the grouped moves: one lane per node for
// schedules with a few moves per node, else 64 x 64 tiles
template <int S>
void moves_writer(const Graph &g, bool lanes, const int32_t *base, int32_t P,
                  const MovesScratch &m, int32_t *lab_w, int64_t lab_stride, int32_t K,
                  int32_t *err, int32_t *fit, uint32_t fit_limit, int l16, const int32_t *gate,
                  int32_t gate_want) {
    const int32_t V = g.V;
    if (lanes)
        k_moves_lanes<S><<<(unsigned)((V + 255) / 256), 256, 0, g.stream>>>(
            V, P, g.order, base, m.off, m.ent, lab_w, lab_stride, K, err, fit, fit_limit, l16,
            gate, gate_want);
    else
        k_moves_to_slices<S><<<(unsigned)((V + 63) / 64), 256, 0, g.stream>>>(
            V, P, g.order, base, m.off, m.ent, lab_w, lab_stride, K, err, fit, fit_limit, l16,
            gate, gate_want);
}

hipError_t launch_moves_writer(const Graph &g, const int32_t *base, int32_t P, int64_t M,
                               int32_t S, const MovesScratch &m, int32_t *lab_w,
                               int64_t lab_stride, int32_t K, int32_t *err, int32_t *fit,
                               uint32_t fit_limit, bool lab16, const int32_t *gate,
                               int32_t gate_want) {
    if (lab16 && (S != 2 || lab_stride % 2 != 0)) return hipErrorInvalidValue;
    const bool lanes = M <= (int64_t)kLaneMovesPerNode * g.V;
    const int l16 = lab16 ? 1 : 0;
    if (S == 1)
        moves_writer<1>(g, lanes, base, P, m, lab_w, lab_stride, K, err, fit, fit_limit, l16,
                        gate, gate_want);
    else if (S == 2)
        moves_writer<2>(g, lanes, base, P, m, lab_w, lab_stride, K, err, fit, fit_limit, l16,
                        gate, gate_want);
    else if (S == 4)
        moves_writer<4>(g, lanes, base, P, m, lab_w, lab_stride, K, err, fit, fit_limit, l16,
                        gate, gate_want);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

}  // namespace

hipError_t launch_moves_to_slices(const Graph &g, const int32_t *base, int32_t P,
                                  const int64_t *step_ptr, int64_t M, const int32_t *node,
                                  const int32_t *label, int32_t S, int32_t *scratch,
                                  int32_t *lab_w, int64_t lab_stride, int32_t K, int32_t *err,
                                  int32_t *fit, uint32_t fit_limit, bool lab16) {
    if (g.V == 0 || P == 0) return hipSuccess;
    if (lab16 && (S != 2 || lab_stride % 2 != 0)) return hipErrorInvalidValue;
    const int32_t V = g.V;
    const MovesScratch m = moves_scratch(V, M, scratch);
    hipError_t e = hipSuccess;
    if (M > 0) {
        k_mv_keys<<<grid_for(M, kBlock), kBlock, 0, g.stream>>>(M, node, V, m.key_in, m.idx_in,
                                                                 err);
        e = hipGetLastError();
        if (e == hipSuccess)
            e = sort_pairs_u32(m.key_in, m.key_out, m.idx_in, m.idx_out, (int32_t)M, 0,
                               (int)mv_key_bits(V), m.temp, g.stream);
    }
    if (e == hipSuccess) {
        k_mv_off<<<grid_for((int64_t)V + 1, kBlock), kBlock, 0, g.stream>>>(V, M, m.key_out,
                                                                            m.off);
        e = hipGetLastError();
    }
    if (e == hipSuccess && M > 0) {
        k_mv_gather<<<grid_for(M, kBlock), kBlock, 0, g.stream>>>(M, P, step_ptr, m.key_out,
                                                                   m.idx_out, label, V, m.ent);
        e = hipGetLastError();
    }
    if (e != hipSuccess) return e;
    return launch_moves_writer(g, base, P, M, S, m, lab_w, lab_stride, K, err, fit, fit_limit,
                               lab16, nullptr, 0);
}

hipError_t launch_moves_write(const Graph &g, const int32_t *base, int32_t P, int64_t M,
                              int32_t S, int32_t *scratch, int32_t *lab_w, int64_t lab_stride,
                              const int32_t *gate, int32_t gate_want) {
    if (g.V == 0 || P == 0) return hipSuccess;
    return launch_moves_writer(g, base, P, M, S, moves_scratch(g.V, M, scratch), lab_w,
                               lab_stride, 0, nullptr, nullptr, kPackLabels, false, gate,
                               gate_want);
}

hipError_t launch_label_memory(const Graph &g, const int32_t *placement, int32_t K,
                               const int64_t *capacity, int64_t *label_mem, int64_t *overflow,
                               int32_t *err) {
    hipError_t e = launch_fill_i64(label_mem, K, 0, g.stream);
    if (e != hipSuccess) return e;
    if (g.V > 0) {
        k_label_sum<<<grid_for(g.V, kBlock, 1024), kBlock, 0, g.stream>>>(g.V, placement, g.mem,
                                                                           K, label_mem, err);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (overflow == nullptr && capacity == nullptr) return hipSuccess;
    return launch_overflow(K, K, capacity, label_mem, overflow, err, g.stream);
}

hipError_t launch_overflow(int64_t n, int32_t K, const int64_t *capacity,
                           const int64_t *label_mem, int64_t *overflow, int32_t *err,
                           hipStream_t s) {
    if (n <= 0) return hipSuccess;
    k_overflow<<<grid_for(n, kBlock), kBlock, 0, s>>>(n, K, capacity, label_mem, overflow, err);
    return hipGetLastError();
}

hipError_t launch_apply_moves(const Graph &g, int32_t *placement, int32_t n, const int32_t *node,
                              const int32_t *label, int32_t *err) {
    if (n <= 0) return hipSuccess;
    const unsigned grid = grid_for(n, kBlock);
    k_moves_mark<<<grid, kBlock, 0, g.stream>>>(n, node, g.V, g.move_stamp, err);
    k_moves_apply<<<grid, kBlock, 0, g.stream>>>(n, node, label, g.V, g.move_stamp, placement,
                                                 err);
    k_moves_reset<<<grid, kBlock, 0, g.stream>>>(n, node, g.V, g.move_stamp);
    return hipGetLastError();
}

namespace {

__global__ void k_check_steps(const int64_t *step_ptr, int32_t P, int64_t M, int32_t *err) {
    for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p <= P;
         p += (int64_t)gridDim.x * blockDim.x) {
        const int64_t x = step_ptr[p];
        const bool bad = (p == 0 && x != 0) || (p == P && x != M) || (p < P && step_ptr[p + 1] < x);
        if (bad) atomicOr(err, kErrSteps);
    }
}

}  // namespace

hipError_t launch_check_steps(const int64_t *step_ptr, int32_t P, int64_t M, int32_t *err,
                              hipStream_t s) {
    if (P < 0) return hipErrorInvalidValue;
    k_check_steps<<<grid_for((int64_t)P + 1, kBlock), kBlock, 0, s>>>(step_ptr, P, M, err);
    return hipGetLastError();
}

// M: the number of moves (the length of node and label), passed by the
// caller; the moves of each step are found by binary search in step_ptr, so
// any step_ptr keeps every access in bounds.
hipError_t launch_build_placements(const Graph &g, const int32_t *base, int32_t P,
                                   const int64_t *step_ptr, int64_t M, const int32_t *node,
                                   const int32_t *label, int32_t *placements, int32_t *err) {
    const int64_t n = (int64_t)g.V * P;
    hipError_t e = launch_fill_i32(placements, n, -1, g.stream);
    if (e != hipSuccess) return e;
    if (M > 0) {
        k_bp_mark<<<grid_for(M, kBlock), kBlock, 0, g.stream>>>(M, P, step_ptr, node, g.V,
                                                                 placements, err);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (g.V > 0 && P > 0) {
        const int waves_per_block = kBlock / kWave;
        k_bp_fill<<<grid_for(g.V, waves_per_block), kBlock, 0, g.stream>>>(g.V, P, base, label,
                                                                            placements);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace pardnn
