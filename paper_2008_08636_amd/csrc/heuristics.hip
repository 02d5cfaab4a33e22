// heuristics.hip -- evaluation of Memory Heuristic II (paper Sec. 3.2.2) for a
// batch of placements.
//
// Node kinds (Sec. 3.2.1): normal nodes (0) hold their output until consumed,
// residual nodes (1) keep their data for the whole run, reference nodes (2)
// mutate a residual node's tensor, reserve nothing and must share its device.
// Per placement p and partition (label) k:
//   res_mem[p][k] = sum of mem(v) over residual v with label k
//   nor_mem[p][k] = sum of mem(v) over normal v with label k
//   balanced[p][k] = Eq. 6 for partition k:
//       K / 2 * (res_mem[k] / RES + nor_mem[k] / NOR) >= 1,
//     a kind with no memory at all counting as the fair share 1 / K,
//     decided exactly in integers;
//   ref_misplaced[p] = number of reference nodes whose target node carries
//     another label.
//
// Design for gfx950: the placements arrive placement-minor, [V][P], so a
// wave reads 64 placements of one node as one 256-byte run. A workgroup owns
// 64 placements and a stripe of nodes, keeps its (placement, label, kind)
// sums in LDS (ds_add_u64) and flushes them with one global atomic per bin;
// a reference node's wave also reads its target's row (again one run) and
// counts mismatches per placement. A second pass decides Eq. 6 per
// (placement, label) with 128-bit integer products.
#include <algorithm>

#include "device_utils.h"
#include "internal.h"

namespace pardnn {

namespace {

constexpr int kCols = 64;          // placements per workgroup
constexpr int kRows = 4;           // nodes in flight per workgroup step (one per wave)
constexpr int kMbLdsLabels = 32;   // labels kept in LDS bins; more go to global atomics

__global__ __launch_bounds__(kCols * kRows) void k_mem_balance_sums(
    int32_t V, int32_t P, int32_t K, const int32_t *placements, const int64_t *mem,
    const int32_t *node_type, const int32_t *ref_target, int64_t *res_mem, int64_t *nor_mem,
    int64_t *misplaced, int32_t *err) {
    __shared__ long long bins[kCols * kMbLdsLabels * 2];   // [col][label][kind]
    __shared__ unsigned long long s_mis[kCols];
    const int col = threadIdx.x % kCols, row = threadIdx.x / kCols;
    const int32_t p = blockIdx.x * kCols + col;
    const bool lds = K <= kMbLdsLabels;
    if (lds)
        for (int i = threadIdx.x; i < kCols * K * 2; i += blockDim.x) bins[i] = 0;
    for (int i = threadIdx.x; i < kCols; i += blockDim.x) s_mis[i] = 0;
    __syncthreads();
    int bad = 0;
    unsigned long long mis = 0;
    const int32_t stripe = (V + gridDim.y - 1) / gridDim.y;
    const int32_t v0 = blockIdx.y * stripe, v1 = min(V, v0 + stripe);
    if (p < P) {
        for (int32_t v = v0 + row; v < v1; v += kRows) {
            const int32_t t = node_type[v];
            const int32_t l = placements[(int64_t)v * P + p];
            if ((uint32_t)l >= (uint32_t)K) {
                bad |= 1;
                continue;
            }
            if (t == 0 || t == 1) {
                const int64_t m = mem[v];
                if (lds)
                    lds_add_i64(&bins[(col * K + l) * 2 + t], m);
                else
                    atomicAdd((unsigned long long *)&(t == 1 ? res_mem : nor_mem)[(int64_t)p * K + l],
                              (unsigned long long)m);
            } else if (t == 2) {
                const int32_t tg = ref_target[v];
                if (tg >= V || tg < -1) {
                    bad |= 4;
                } else if (tg >= 0) {
                    mis += placements[(int64_t)tg * P + p] != l;
                }
            } else {
                bad |= 2;
            }
        }
    }
    if (bad) atomicOr(err, bad);
    if (mis) atomicAdd(&s_mis[col], mis);
    __syncthreads();
    if (threadIdx.x < kCols && p < P && s_mis[threadIdx.x])
        atomicAdd((unsigned long long *)&misplaced[p], s_mis[threadIdx.x]);
    if (lds) {
        for (int i = threadIdx.x; i < kCols * K * 2; i += blockDim.x) {
            const int c = i / (K * 2), l = (i / 2) % K, kind = i % 2;
            const int32_t pc = blockIdx.x * kCols + c;
            if (pc < P && bins[i] != 0)
                atomicAdd((unsigned long long *)&(kind == 1 ? res_mem : nor_mem)[(int64_t)pc * K + l],
                          (unsigned long long)bins[i]);
        }
    }
}

// 128-bit unsigned values as two 64-bit halves
struct U128 {
    uint64_t hi, lo;
};
__device__ __forceinline__ U128 mul64(uint64_t a, uint64_t b) { return {__umul64hi(a, b), a * b}; }
__device__ __forceinline__ U128 add128(U128 a, U128 b) {
    const uint64_t lo = a.lo + b.lo;
    return {a.hi + b.hi + (lo < a.lo ? 1u : 0u), lo};
}
__device__ __forceinline__ bool ge128(U128 a, U128 b) {
    return a.hi > b.hi || (a.hi == b.hi && a.lo >= b.lo);
}
// ceil(a / d) for d in [1, 2^32): long division over 32-bit limbs
__device__ __forceinline__ U128 ceil_div128(U128 a, uint32_t d) {
    const uint32_t limb[4] = {(uint32_t)(a.hi >> 32), (uint32_t)a.hi, (uint32_t)(a.lo >> 32),
                              (uint32_t)a.lo};
    uint32_t q[4];
    uint64_t rem = 0;
    for (int i = 0; i < 4; i++) {
        const uint64_t cur = (rem << 32) | limb[i];
        q[i] = (uint32_t)(cur / d);
        rem = cur % d;
    }
    U128 r = {((uint64_t)q[0] << 32) | q[1], ((uint64_t)q[2] << 32) | q[3]};
    if (rem != 0) r = add128(r, U128{0, 1});
    return r;
}

// Eq. 6 per (placement, label): one thread per placement.
__global__ void k_mem_balance_decide(int32_t P, int32_t K, const int64_t *res_mem,
                                     const int64_t *nor_mem, uint8_t *balanced) {
    for (int32_t p = blockIdx.x * blockDim.x + threadIdx.x; p < P; p += gridDim.x * blockDim.x) {
        const int64_t *rs = res_mem + (int64_t)p * K;
        const int64_t *ns = nor_mem + (int64_t)p * K;
        uint64_t RES = 0, NOR = 0;
        for (int32_t k = 0; k < K; k++) {
            RES += (uint64_t)rs[k];
            NOR += (uint64_t)ns[k];
        }
        for (int32_t k = 0; k < K; k++) {
            const uint64_t r = (uint64_t)rs[k], n = (uint64_t)ns[k];
            bool ok;
            if (RES == 0 && NOR == 0) {
                ok = true;
            } else if (RES == 0) {   // 1/K + n/NOR >= 2/K  <=>  K n >= NOR
                ok = ge128(mul64((uint64_t)K, n), U128{0, NOR});
            } else if (NOR == 0) {
                ok = ge128(mul64((uint64_t)K, r), U128{0, RES});
            } else {   // K (r NOR + n RES) >= 2 RES NOR  <=>  r NOR + n RES >= ceil(2 RES NOR / K)
                const U128 x = add128(mul64(r, NOR), mul64(n, RES));
                const U128 rn = mul64(RES, NOR);
                const U128 two = add128(rn, rn);
                ok = ge128(x, ceil_div128(two, (uint32_t)K));
            }
            balanced[(int64_t)p * K + k] = ok ? 1 : 0;
        }
    }
}

}  // namespace

hipError_t launch_mem_balance(const Graph &g, int32_t P, const int32_t *placements,
                              const int32_t *node_type, const int32_t *ref_target, int32_t K,
                              int64_t *res_mem, int64_t *nor_mem, uint8_t *balanced,
                              int64_t *misplaced, int32_t *err) {
    hipError_t e = launch_fill_i64(res_mem, (int64_t)P * K, 0, g.stream);
    if (e == hipSuccess) e = launch_fill_i64(nor_mem, (int64_t)P * K, 0, g.stream);
    if (e == hipSuccess) e = launch_fill_i64(misplaced, P, 0, g.stream);
    if (e != hipSuccess) return e;
    if (g.V > 0) {
        // enough workgroups to fill the chip: placement tiles x node stripes
        const int32_t tiles = (P + kCols - 1) / kCols;
        int32_t stripes = (1024 + tiles - 1) / tiles;
        stripes = std::max(1, std::min(stripes, (g.V + 255) / 256));
        k_mem_balance_sums<<<dim3((unsigned)tiles, (unsigned)stripes), kCols * kRows, 0,
                             g.stream>>>(g.V, P, K, placements, g.mem, node_type, ref_target,
                                         res_mem, nor_mem, misplaced, err);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    k_mem_balance_decide<<<(unsigned)((P + 255) / 256), 256, 0, g.stream>>>(P, K, res_mem, nor_mem,
                                                                          balanced);
    return hipGetLastError();
}

}  // namespace pardnn
