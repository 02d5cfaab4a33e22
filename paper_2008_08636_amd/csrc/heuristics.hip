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
// wave reads 64 placements of one node as one 256-byte run, eight nodes' runs
// in flight at once. A workgroup owns 64 placements and a stripe of nodes,
// keeps its (label, kind, placement) sums in LDS (ds_add_u64 on 64
// consecutive bins per wave, free of bank conflicts) and flushes them with one
// global atomic per bin;
// a reference node's wave also reads its target's row (again one run) and
// counts mismatches per placement. A second pass decides Eq. 6 per
// (placement, label) with 128-bit integer products.
#include <algorithm>

#include "device_utils.h"
#include "internal.h"

namespace pardnn {

namespace {

constexpr int kCols = 64;          // placements per workgroup
constexpr int kRows = 4;           // node rows in flight per workgroup step (one per wave)
constexpr int kUnroll = 8;         // nodes per wave whose placement loads are issued together
constexpr int kMbLdsLabels = 32;   // labels kept in LDS bins; more go to global atomics

template <bool LDS>
__global__ __launch_bounds__(kCols * kRows) void k_mem_balance_sums(
    int32_t V, int32_t P, int32_t K, const int32_t *__restrict__ placements,
    const int64_t *__restrict__ mem, const int32_t *__restrict__ node_type,
    const int32_t *__restrict__ ref_target, int64_t *__restrict__ res_mem,
    int64_t *__restrict__ nor_mem, int64_t *__restrict__ misplaced, int32_t *__restrict__ err) {
    // LDS bins [label][kind][col] plus one trash row for out-of-range labels:
    // the 64 lanes of a wave (64 placements) add to 64 consecutive 8-byte
    // bins, so an LDS atomic never conflicts on a bank (dynamic LDS,
    // (2 K + 1) * kCols entries)
    extern __shared__ long long bins[];
    __shared__ unsigned long long s_mis[kCols];
    // logical (tile, stripe): the placement tiles of one node stripe run on
    // one XCD, so the 128-byte lines that two neighbouring tiles share are
    // fetched into one L2 only
    const int32_t tiles = (P + kCols - 1) / kCols;
    const int32_t lb = xcd_major(blockIdx.x, gridDim.x);
    const int32_t tile = lb % tiles, stripe_id = lb / tiles, n_stripes = gridDim.x / tiles;
    const int col = threadIdx.x % kCols;
    const int row = __builtin_amdgcn_readfirstlane(threadIdx.x / kCols);
    const int32_t p = tile * kCols + col;
    if (LDS)
        for (int i = threadIdx.x; i < (2 * K + 1) * kCols; i += blockDim.x) bins[i] = 0;
    for (int i = threadIdx.x; i < kCols; i += blockDim.x) s_mis[i] = 0;
    __syncthreads();
    int bad = 0;
    unsigned long long mis = 0;
    const int32_t stripe = (V + n_stripes - 1) / n_stripes;
    const int32_t v0 = stripe_id * stripe, v1 = min(V, v0 + stripe);
    // one node's contribution to this lane's placement; t, m and tg are the
    // node's kind, memory and target (wave-uniform), l its label here
    auto account = [&](int32_t t, int64_t m, int32_t tg, int32_t l) {
        const bool ok = (uint32_t)l < (uint32_t)K;
        bad |= ok ? 0 : 1;
        if (t == 0 || t == 1) {
            if (LDS) {
                lds_add_i64(&bins[(ok ? (l * 2 + t) : 2 * K) * kCols + col], m);
            } else if (ok) {
                atomicAdd((unsigned long long *)&(t == 1 ? res_mem : nor_mem)[(int64_t)p * K + l],
                          (unsigned long long)m);
            }
        } else if (t == 2) {
            if (tg >= V || tg < -1)
                bad |= 4;
            else if (tg >= 0)
                mis += placements[(int64_t)tg * P + p] != l;
        } else {
            bad |= 2;
        }
    };
    if (p < P) {
        // Node indices are wave-uniform, so node records come through scalar
        // loads. Software-pipelined: the kUnroll placement runs and records
        // of the next group are issued before the current group is added up
        // (indices clamped into the graph, so the look-ahead stays in bounds).
        struct Group {
            int32_t t[kUnroll], l[kUnroll], tg[kUnroll];
            int64_t m[kUnroll];
        };
        auto fetch = [&](int32_t v, Group &G) {
#pragma unroll
            for (int u = 0; u < kUnroll; u++) {
                const int32_t vs = __builtin_amdgcn_readfirstlane(min(v + u * kRows, V - 1));
                G.l[u] = placements[(int64_t)vs * P + p];
                G.t[u] = node_type[vs];
                G.m[u] = mem[vs];
                G.tg[u] = ref_target[vs];
            }
        };
        int32_t v = v0 + row;
        if (v + (kUnroll - 1) * kRows < v1) {
            Group cur, nxt;
            fetch(v, cur);
            while (true) {
                const int32_t vn = v + kUnroll * kRows;
                fetch(vn, nxt);
#pragma unroll
                for (int u = 0; u < kUnroll; u++)
                    account(__builtin_amdgcn_readfirstlane(cur.t[u]), cur.m[u],
                            __builtin_amdgcn_readfirstlane(cur.tg[u]), cur.l[u]);
                v = vn;
                if (v + (kUnroll - 1) * kRows >= v1) break;
                cur = nxt;
            }
        }
        for (; v < v1; v += kRows) {
            const int32_t vs = __builtin_amdgcn_readfirstlane(v);
            account(node_type[vs], mem[vs], ref_target[vs], placements[(int64_t)vs * P + p]);
        }
    }
    if (bad) atomicOr(err, bad);
    if (mis) atomicAdd(&s_mis[col], mis);
    __syncthreads();
    if (threadIdx.x < kCols && p < P && s_mis[threadIdx.x])
        atomicAdd((unsigned long long *)&misplaced[p], s_mis[threadIdx.x]);
    if (LDS) {
        for (int i = threadIdx.x; i < kCols * K * 2; i += blockDim.x) {
            const int c = i % kCols, kind = (i / kCols) % 2, l = i / (2 * kCols);
            const int32_t pc = tile * kCols + c;
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
        int32_t stripes = (2048 + tiles - 1) / tiles;
        stripes = std::max(1, std::min(stripes, (g.V + 255) / 256));
        const unsigned grid = (unsigned)tiles * (unsigned)stripes;   // tile-minor, see xcd_major
        if (g.timing) (void)hipEventRecord(g.ev0, g.stream);
        if (K <= kMbLdsLabels)
            k_mem_balance_sums<true>
                <<<grid, kCols * kRows, (size_t)(2 * K + 1) * kCols * sizeof(long long),
                   g.stream>>>(g.V, P, K, placements, g.mem, node_type, ref_target, res_mem,
                               nor_mem, misplaced, err);
        else
            k_mem_balance_sums<false><<<grid, kCols * kRows, 0, g.stream>>>(
                g.V, P, K, placements, g.mem, node_type, ref_target, res_mem, nor_mem,
                misplaced, err);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if (g.timing) (void)hipEventRecord(g.ev1, g.stream);
    }
    k_mem_balance_decide<<<(unsigned)((P + 255) / 256), 256, 0, g.stream>>>(P, K, res_mem, nor_mem,
                                                                          balanced);
    return hipGetLastError();
}

}  // namespace pardnn
