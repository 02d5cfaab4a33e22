// structure.hip -- graph ingest: validation, degree counts, scans and the
// CSR/CSC builds in the original and in the level-major numbering.
//
// Validation bounds every path length by sum(comp) + sum(edge_cost) (paper,
// Table 2: a path's length sums comp over its nodes and comm over its edges),
// so one exact check at ingest rules out int64 overflow in every later kernel.
#include "device_utils.h"
#include "internal.h"

namespace pardnn {

namespace {

constexpr int kBlock = 256;
constexpr int kScanThreads = 1024;
constexpr int kScanItems = 4;
constexpr int kScanTile = kScanThreads * kScanItems;

inline unsigned grid_for(int64_t n, int block, int cap = 65536) {
    int64_t g = (n + block - 1) / block;
    if (g < 1) g = 1;
    if (g > cap) g = cap;
    return (unsigned)g;
}

__global__ void k_fill_i32(int32_t *p, int64_t n, int32_t value) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = value;
}

__global__ void k_fill_i64(int64_t *p, int64_t n, int64_t value) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = value;
}

// Range and sign checks plus exact sums split at bit 32: with fewer than 2^32
// non-negative int64 terms, the low halves sum below 2^64 and the high halves
// below 2^63, so neither accumulator can wrap.
__global__ void k_validate(int32_t V, int64_t E, const int32_t *src, const int32_t *dst,
                           const int64_t *comp, const int64_t *cost, const int64_t *mem,
                           ValidateAcc *acc) {
    unsigned long long flags = 0, wlo = 0, whi = 0, mlo = 0, mhi = 0;
    const int64_t n = V > E ? (int64_t)V : E;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        if (i < E) {
            int32_t s = src[i], d = dst[i];
            if (s < 0 || s >= V || d < 0 || d >= V) flags |= 1ull;
            int64_t c = cost[i];
            if (c < 0) {
                flags |= 2ull;
            } else {
                wlo += (unsigned long long)c & 0xffffffffull;
                whi += (unsigned long long)c >> 32;
            }
        }
        if (i < V) {
            int64_t c = comp[i], m = mem[i];
            if (c < 0 || m < 0) {
                flags |= 2ull;
            } else {
                wlo += (unsigned long long)c & 0xffffffffull;
                whi += (unsigned long long)c >> 32;
                mlo += (unsigned long long)m & 0xffffffffull;
                mhi += (unsigned long long)m >> 32;
            }
        }
    }
    wlo = wave_sum_u64(wlo);
    whi = wave_sum_u64(whi);
    mlo = wave_sum_u64(mlo);
    mhi = wave_sum_u64(mhi);
    // OR-reduce the flags across the wave
    for (int off = kWave / 2; off > 0; off >>= 1) flags |= __shfl_xor(flags, off, kWave);
    if (lane_id() == 0) {
        if (flags) atomicOr(&acc->flags, flags);
        atomicAdd(&acc->w_lo, wlo);
        atomicAdd(&acc->w_hi, whi);
        atomicAdd(&acc->m_lo, mlo);
        atomicAdd(&acc->m_hi, mhi);
    }
}

__global__ void k_count_degrees(int64_t E, const int32_t *src, const int32_t *dst,
                                int32_t *outdeg, int32_t *indeg) {
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < E;
         e += (int64_t)gridDim.x * blockDim.x) {
        atomicAdd(&outdeg[src[e]], 1);
        atomicAdd(&indeg[dst[e]], 1);
    }
}

// ---- three-pass exclusive scan of int32 counts (totals < 2^31) ----

__global__ __launch_bounds__(kScanThreads) void k_scan_tile_sums(const int32_t *in, int32_t n,
                                                                  int32_t *tile_sums) {
    __shared__ int wsum[kScanThreads / kWave + 1];
    const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
    int s = 0;
#pragma unroll
    for (int j = 0; j < kScanItems; j++)
        if (base + j < n) s += in[base + j];
    int total;
    block_excl_scan_i32(s, wsum, &total);
    if (threadIdx.x == 0) tile_sums[blockIdx.x] = total;
}

__global__ __launch_bounds__(kScanThreads) void k_scan_tile_offsets(int32_t *tile_sums,
                                                                     int32_t n_tiles,
                                                                     int32_t *out, int32_t n) {
    __shared__ int wsum[kScanThreads / kWave + 1];
    int carry = 0;
    for (int32_t b = 0; b < n_tiles; b += kScanThreads) {
        int32_t i = b + threadIdx.x;
        int x = i < n_tiles ? tile_sums[i] : 0;
        int total;
        int ex = block_excl_scan_i32(x, wsum, &total);
        if (i < n_tiles) tile_sums[i] = carry + ex;
        carry += total;
        __syncthreads();
    }
    if (threadIdx.x == 0) out[n] = carry;
}

__global__ __launch_bounds__(kScanThreads) void k_scan_apply(const int32_t *in, int32_t n,
                                                             const int32_t *tile_offsets,
                                                             int32_t *out) {
    __shared__ int wsum[kScanThreads / kWave + 1];
    const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
    int v[kScanItems];
    int s = 0;
#pragma unroll
    for (int j = 0; j < kScanItems; j++) {
        v[j] = base + j < n ? in[base + j] : 0;
        s += v[j];
    }
    int total;
    int ex = block_excl_scan_i32(s, wsum, &total) + tile_offsets[blockIdx.x];
#pragma unroll
    for (int j = 0; j < kScanItems; j++) {
        if (base + j < n) out[base + j] = ex;
        ex += v[j];
    }
}

__global__ void k_scatter_orig_csr(int64_t E, const int32_t *src, const int32_t *dst,
                                   int32_t *cursor, int32_t *o_nbr) {
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < E;
         e += (int64_t)gridDim.x * blockDim.x) {
        int32_t pos = atomicAdd(&cursor[src[e]], 1);
        o_nbr[pos] = dst[e];
    }
}

__global__ void k_rank_and_permute(int32_t V, const int32_t *order, const int32_t *indeg,
                                   const int32_t *outdeg, const int64_t *comp,
                                   const int64_t *mem, int32_t *rank, int32_t *indeg_lm,
                                   int32_t *outdeg_lm, int64_t *comp_lm, int64_t *mem_lm) {
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < V; i += gridDim.x * blockDim.x) {
        int32_t v = order[i];
        rank[v] = i;
        indeg_lm[i] = indeg[v];
        outdeg_lm[i] = outdeg[v];
        comp_lm[i] = comp[v];
        mem_lm[i] = mem[v];
    }
}

__global__ void k_scatter_lm(int64_t E, const int32_t *src, const int32_t *dst,
                             const int64_t *cost, const int32_t *rank, int32_t *cin,
                             int32_t *cout, int32_t *in_src, int32_t *in_dst, int64_t *in_cost,
                             int32_t *out_src, int32_t *out_dst, int32_t *out_dst_orig,
                             int64_t *out_cost) {
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < E;
         e += (int64_t)gridDim.x * blockDim.x) {
        int32_t so = src[e], d = dst[e];
        int32_t u = rank[so], v = rank[d];
        int64_t c = cost[e];
        int32_t pi = atomicAdd(&cin[v], 1);
        in_src[pi] = u;
        in_dst[pi] = v;
        in_cost[pi] = c;
        int32_t po = atomicAdd(&cout[u], 1);
        out_src[po] = u;
        out_dst[po] = v;
        out_dst_orig[po] = d;
        out_cost[po] = c;
    }
}

__global__ void k_pack_records(int64_t E, int32_t V, const int32_t *in_src,
                               const int32_t *in_dst, const int64_t *in_cost,
                               const int32_t *out_src, const int32_t *out_dst,
                               const int64_t *out_cost, const int64_t *comp_lm,
                               const int64_t *mem_lm, EdgeRec16 *in_rec, EdgeRec16 *out_rec,
                               NodeRec16 *node_rec) {
    const int64_t n = E > V ? E : (int64_t)V;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        if (i < E) {
            in_rec[i] = EdgeRec16{in_src[i], in_dst[i], in_cost[i]};
            out_rec[i] = EdgeRec16{out_dst[i], out_src[i], out_cost[i]};
        }
        if (i < V) node_rec[i] = NodeRec16{comp_lm[i], mem_lm[i]};
    }
}

__global__ void k_level_info(int32_t L, const int32_t *level_ptr, const int32_t *in_off,
                             const int32_t *out_off, LevelInfo *linfo) {
    // entries 0..L, and L + 1 repeating L (the empty level past either end)
    for (int32_t k = blockIdx.x * blockDim.x + threadIdx.x; k <= L + 1; k += gridDim.x * blockDim.x) {
        int32_t lo = level_ptr[min(k, L)];
        LevelInfo li;
        li.node_lo = lo;
        li.in_e_lo = in_off[lo];
        li.out_e_lo = out_off[lo];
        li.pad = 0;
        linfo[k] = li;
    }
}

}  // namespace

hipError_t launch_fill_i32(int32_t *p, int64_t n, int32_t value, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    k_fill_i32<<<grid_for(n, kBlock), kBlock, 0, s>>>(p, n, value);
    return hipGetLastError();
}

__global__ void k_iota_i32(int32_t *p, int32_t n) {
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x)
        p[i] = i;
}

hipError_t launch_iota_i32(int32_t *p, int32_t n, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    k_iota_i32<<<grid_for(n, kBlock), kBlock, 0, s>>>(p, n);
    return hipGetLastError();
}

hipError_t launch_fill_i64(int64_t *p, int64_t n, int64_t value, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    k_fill_i64<<<grid_for(n, kBlock), kBlock, 0, s>>>(p, n, value);
    return hipGetLastError();
}

hipError_t launch_validate(const Graph &g, const int32_t *src, const int32_t *dst,
                           const int64_t *comp, const int64_t *cost, const int64_t *mem,
                           ValidateAcc *acc) {
    int64_t n = g.V > g.E ? (int64_t)g.V : g.E;
    k_validate<<<grid_for(n, kBlock, 4096), kBlock, 0, g.stream>>>(g.V, g.E, src, dst, comp,
                                                                    cost, mem, acc);
    return hipGetLastError();
}

hipError_t launch_count_degrees(const Graph &g) {
    if (g.E == 0) return hipSuccess;
    k_count_degrees<<<grid_for(g.E, kBlock), kBlock, 0, g.stream>>>(g.E, g.e_src, g.e_dst,
                                                                     g.outdeg, g.indeg);
    return hipGetLastError();
}

size_t scan_workspace_elems(int32_t n) { return (size_t)(n / kScanTile + 2); }

// out[0..n) = exclusive prefix sums of in[0..n), out[n] = total. `ws` holds
// scan_workspace_elems(n) ints.
hipError_t launch_exclusive_scan(const int32_t *in, int32_t *out, int32_t n, int32_t *ws,
                                 hipStream_t s) {
    int32_t tiles = (n + kScanTile - 1) / kScanTile;
    if (tiles < 1) tiles = 1;
    k_scan_tile_sums<<<tiles, kScanThreads, 0, s>>>(in, n, ws);
    k_scan_tile_offsets<<<1, kScanThreads, 0, s>>>(ws, tiles, out, n);
    k_scan_apply<<<tiles, kScanThreads, 0, s>>>(in, n, ws, out);
    return hipGetLastError();
}

hipError_t launch_build_orig_csr(const Graph &g, int32_t *cursor) {
    hipError_t err = hipMemcpyAsync(cursor, g.o_off, sizeof(int32_t) * (size_t)g.V,
                                    hipMemcpyDeviceToDevice, g.stream);
    if (err != hipSuccess) return err;
    if (g.E == 0) return hipSuccess;
    k_scatter_orig_csr<<<grid_for(g.E, kBlock), kBlock, 0, g.stream>>>(g.E, g.e_src, g.e_dst,
                                                                        cursor, g.o_nbr);
    return hipGetLastError();
}

// Level-major CSC and CSR: rank = inverse of order, per-node degrees in lm
// order, scans, then one scatter of the edge list into both.
hipError_t launch_build_lm(Graph &g, int32_t *deg_ws, int32_t *cursor_in, int32_t *cursor_out,
                           int32_t *scan_ws) {
    const int32_t V = g.V;
    int32_t *indeg_lm = deg_ws, *outdeg_lm = deg_ws + V;
    k_rank_and_permute<<<grid_for(V, kBlock), kBlock, 0, g.stream>>>(
        V, g.order, g.indeg, g.outdeg, g.comp, g.mem, g.rank, indeg_lm, outdeg_lm, g.comp_lm,
        g.mem_lm);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    if ((err = launch_fill_i32(g.rank + V, 1, -1, g.stream)) != hipSuccess) return err;
    if ((err = launch_exclusive_scan(indeg_lm, g.in_off, V, scan_ws, g.stream)) != hipSuccess)
        return err;
    if ((err = launch_exclusive_scan(outdeg_lm, g.out_off, V, scan_ws, g.stream)) != hipSuccess)
        return err;
    if ((err = hipMemcpyAsync(cursor_in, g.in_off, sizeof(int32_t) * (size_t)V,
                              hipMemcpyDeviceToDevice, g.stream)) != hipSuccess)
        return err;
    if ((err = hipMemcpyAsync(cursor_out, g.out_off, sizeof(int32_t) * (size_t)V,
                              hipMemcpyDeviceToDevice, g.stream)) != hipSuccess)
        return err;
    if (g.E > 0) {
        k_scatter_lm<<<grid_for(g.E, kBlock), kBlock, 0, g.stream>>>(
            g.E, g.e_src, g.e_dst, g.e_cost, g.rank, cursor_in, cursor_out, g.in_src, g.in_dst,
            g.in_cost, g.out_src, g.out_dst, g.out_dst_orig, g.out_cost);
        if ((err = hipGetLastError()) != hipSuccess) return err;
    }
    const int64_t nrec = g.E > g.V ? g.E : (int64_t)g.V;
    if (nrec > 0) {
        k_pack_records<<<grid_for(nrec, kBlock), kBlock, 0, g.stream>>>(
            g.E, g.V, g.in_src, g.in_dst, g.in_cost, g.out_src, g.out_dst, g.out_cost, g.comp_lm,
            g.mem_lm, g.in_rec, g.out_rec, g.node_rec);
        if ((err = hipGetLastError()) != hipSuccess) return err;
    }
    k_level_info<<<grid_for(g.L + 2, kBlock), kBlock, 0, g.stream>>>(g.L, g.level_ptr, g.in_off,
                                                                      g.out_off, g.linfo);
    return hipGetLastError();
}

}  // namespace pardnn
