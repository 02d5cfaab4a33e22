// sweep_common.h -- value encodings and addressing shared by the sweep kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>

namespace pardnn {

// Element idx of an array whose base pointer is uniform over the wave,
// addressed with a 32-bit byte offset, so that the access uses the scalar base
// + 32-bit vector offset form: no 64-bit index arithmetic and no register pair
// holding a sign-extended index. Graph creation bounds V and E so that every
// such offset stays below 2^32.
template <class T>
__device__ __forceinline__ T &at(T *base, uint32_t idx) {
    using B = typename std::conditional<std::is_const<T>::value, const char, char>::type;
    return *reinterpret_cast<T *>(reinterpret_cast<B *>(base) + idx * (uint32_t)sizeof(T));
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

}  // namespace pardnn
