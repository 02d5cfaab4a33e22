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
#include "device_utils.h"
#include "internal.h"

namespace pardnn {

namespace {

constexpr int kBlock = 256;
constexpr int kLdsBins = 4096;

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

// Labels of successive placements straight into the sweep's slice-major
// workspace lab_w[slice][v][s] (v level-major, placement p = slice * S + s).
// `mat` holds, per original node row, the index of the last move at each step
// (k_bp_mark) or -1. A workgroup owns 64 consecutive level-major nodes and
// walks the placements in chunks of 64: one wave scans one node row chunk
// (coalesced), carrying the running label across chunks, into an LDS tile
// that is then written out slice by slice as contiguous runs.
template <int S>
__global__ __launch_bounds__(256) void k_moves_to_slices(int32_t V, int32_t P,
                                                         const int32_t *order,
                                                         const int32_t *base,
                                                         const int32_t *label,
                                                         const int32_t *mat, int32_t *lab_w,
                                                         int64_t lab_stride, int32_t K,
                                                         int32_t *err) {
    constexpr int TV = 64, TP = 64;
    __shared__ int32_t tile[TV][TP + 1];
    __shared__ int32_t carry[TV];
    __shared__ int32_t rows[TV];
    const int lane = lane_id(), w = wave_id();
    const int32_t v0 = blockIdx.x * TV;
    const int32_t n_slices = (P + S - 1) / S;
    for (int r = threadIdx.x; r < TV; r += 256) {
        const int32_t v = v0 + r;
        rows[r] = v < V ? order[v] : -1;
        carry[r] = v < V ? base[order[v]] : 0;
    }
    __syncthreads();
    constexpr int RW = TV / (256 / kWave);  // node rows per wave
    for (int32_t c0 = 0; c0 < n_slices * S; c0 += TP) {
        // all of this wave's row chunks in flight at once, then scan each
        const int32_t p = c0 + lane;
        int32_t m[RW];
#pragma unroll
        for (int j = 0; j < RW; j++) {
            const int32_t o = rows[w + j * (256 / kWave)];
            m[j] = mat[(int64_t)(o >= 0 ? o : 0) * P + min(p, P - 1)];
            if (o < 0 || p >= P) m[j] = -1;
        }
        int32_t mm[RW], last[RW];
#pragma unroll
        for (int j = 0; j < RW; j++) {
            int32_t l = m[j] >= 0 ? lane : -1;
#pragma unroll
            for (int off = 1; off < kWave; off <<= 1) {
                int32_t y = __shfl_up(l, off, kWave);
                if (lane >= off) l = max(l, y);
            }
            last[j] = l;
            mm[j] = __shfl(m[j], l < 0 ? 0 : l, kWave);
        }
        int32_t lv[RW];
#pragma unroll
        for (int j = 0; j < RW; j++) lv[j] = label[last[j] >= 0 ? mm[j] : 0];
#pragma unroll
        for (int j = 0; j < RW; j++) {
            const int r = w + j * (256 / kWave);
            const int32_t val = last[j] >= 0 ? lv[j] : carry[r];
            tile[r][lane] = val;
            const int32_t tail = __shfl(val, kWave - 1, kWave);
            if (lane == 0) carry[r] = tail;
        }
        __syncthreads();
        const int32_t sl0 = c0 / S;
        const int n_sl = min(TP / S, n_slices - sl0);
        for (int i = threadIdx.x; i < n_sl * TV * S; i += 256) {
            const int sl = i / (TV * S), j = i % (TV * S);
            const int r = j / S, s2 = j % S;
            const int32_t v = v0 + r;
            if (v < V) {
                const int32_t x = tile[r][sl * S + s2];
                lab_w[(int64_t)(sl0 + sl) * lab_stride + (int64_t)v * S + s2] = x;
                if (K > 0 && (x < 0 || x >= K) && c0 + sl * S + s2 < P) atomicOr(err, 1);
            }
        }
        __syncthreads();
    }
}

}  // namespace

hipError_t launch_moves_to_slices(const Graph &g, const int32_t *base, int32_t P,
                                  const int64_t *step_ptr, int64_t M, const int32_t *node,
                                  const int32_t *label, int32_t S, int32_t *mat, int32_t *lab_w,
                                  int64_t lab_stride, int32_t K, int32_t *err) {
    if (g.V == 0 || P == 0) return hipSuccess;
    hipError_t e = launch_fill_i32(mat, (int64_t)g.V * P, -1, g.stream);
    if (e != hipSuccess) return e;
    if (M > 0) {
        k_bp_mark<<<grid_for(M, kBlock), kBlock, 0, g.stream>>>(M, P, step_ptr, node, g.V, mat,
                                                                 err);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    const unsigned grid = (unsigned)((g.V + 63) / 64);
    // the label gather is unconditional; without moves it reads a valid dummy
    const int32_t *lab_src = M > 0 ? label : base;
    if (S == 1)
        k_moves_to_slices<1><<<grid, 256, 0, g.stream>>>(g.V, P, g.order, base, lab_src, mat,
                                                         lab_w, lab_stride, K, err);
    else if (S == 2)
        k_moves_to_slices<2><<<grid, 256, 0, g.stream>>>(g.V, P, g.order, base, lab_src, mat,
                                                         lab_w, lab_stride, K, err);
    else if (S == 4)
        k_moves_to_slices<4><<<grid, 256, 0, g.stream>>>(g.V, P, g.order, base, lab_src, mat,
                                                         lab_w, lab_stride, K, err);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
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

// M = step_ptr[P], the number of moves, read on the host by the caller.
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
