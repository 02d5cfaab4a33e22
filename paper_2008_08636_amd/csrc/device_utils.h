// device_utils.h -- wave64 / workgroup primitives shared by the kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace pardnn {

constexpr int kWave = 64;

__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }
__device__ __forceinline__ int wave_id() { return threadIdx.x / kWave; }

// Workgroup-scope relaxed atomics on LDS (ds_max_i64, ds_min_u64, ds_add_u64 ...).
__device__ __forceinline__ void lds_max_i64(long long *p, long long v) {
    __hip_atomic_fetch_max(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ void lds_min_u64(unsigned long long *p, unsigned long long v) {
    __hip_atomic_fetch_min(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ void lds_min_i32(int *p, int v) {
    __hip_atomic_fetch_min(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ void lds_add_i64(long long *p, long long v) {
    __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

__device__ __forceinline__ int wave_incl_scan_i32(int v) {
    const int lane = lane_id();
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        int y = __shfl_up(v, off, kWave);
        if (lane >= off) v += y;
    }
    return v;
}

__device__ __forceinline__ long long wave_max_i64(long long v) {
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) {
        long long y = __shfl_xor(v, off, kWave);
        v = y > v ? y : v;
    }
    return v;
}

__device__ __forceinline__ unsigned long long wave_sum_u64(unsigned long long v) {
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
    return v;
}

// Exclusive scan of one int per thread over the workgroup. `wsum` is LDS of
// at least blockDim.x / 64 + 1 ints. Every thread receives the total.
// Contains two barriers; the caller must barrier before reusing `wsum`.
__device__ __forceinline__ int block_excl_scan_i32(int x, int *wsum, int *total) {
    const int lane = lane_id(), wid = wave_id();
    const int nw = blockDim.x / kWave;
    int incl = wave_incl_scan_i32(x);
    if (lane == kWave - 1) wsum[wid] = incl;
    __syncthreads();
    if (wid == 0) {
        int w = lane < nw ? wsum[lane] : 0;
        int wi = wave_incl_scan_i32(w);
        if (lane < nw) wsum[lane] = wi;
    }
    __syncthreads();
    *total = wsum[nw - 1];
    int base = wid > 0 ? wsum[wid - 1] : 0;
    return base + incl - x;
}

// Workgroup b of n runs on XCD b % 8 (round-robin dispatch); this maps b to a
// logical index such that the workgroups of one XCD take consecutive logical
// indices (a bijection on [0, n)), so neighbouring work shares one L2.
__device__ __forceinline__ int32_t xcd_major(int32_t b, int32_t n) {
    constexpr int kXcd = 8;
    const int32_t x = b % kXcd;
    int32_t start = 0;
    for (int32_t y = 0; y < x; y++) start += (n - y + kXcd - 1) / kXcd;
    return start + b / kXcd;
}

}  // namespace pardnn
