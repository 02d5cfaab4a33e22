// radix_sort.hip -- stable LSD radix sort of (key, int32 value) pairs and an
// int64 prefix scan, written for gfx950; they order the levels (level, id),
// group refinement moves by node, rank clusters by criticality and build the
// span-work tables.
//
// One pass per 8-bit digit, three launches per pass:
//   k_rs_hist     each tile of 2048 keys counts its digits (LDS bins) and
//                 writes them digit-major: counts[digit][tile];
//   scan          an exclusive scan of that matrix gives, for every (digit,
//                 tile), the first output position of the tile's keys with
//                 that digit -- earlier digits first, then earlier tiles;
//   k_rs_scatter  each tile ranks its keys stably inside the tile and writes
//                 them out.
// Stable ranking inside a tile without per-thread digit counters: every wave
// owns a contiguous run of 512 keys, read as 8 rows of 64 lanes (lane-minor,
// so a row is input order). Row by row, the lanes holding one digit find each
// other with one ballot per digit bit (their "peer" mask); a lane's rank among
// its peers is the popcount of the peers below it, and the lowest peer adds
// the group's size to the wave's running count of that digit in LDS. The wave
// counts are then prefixed over the waves and the digits, the tile is
// rearranged in LDS into digit order, and written out in runs: consecutive
// threads write consecutive positions of one digit's run.
#include "device_utils.h"
#include "internal.h"

namespace pardnn {

namespace {

constexpr int kRsThreads = 256;
constexpr int kRsItems = 8;                          // keys per thread
constexpr int kRsTile = kRsThreads * kRsItems;       // 2048 keys per tile
constexpr int kRsWaves = kRsThreads / kWave;         // 4
constexpr int kRsWaveKeys = kWave * kRsItems;        // 512 keys per wave
constexpr int kRsBits = 8;
constexpr int kRsBins = 1 << kRsBits;                // 256
static_assert(kRsBins == kRsThreads, "one digit per thread in the prefix steps");

inline size_t al256(size_t b) { return (b + 255) / 256 * 256; }

inline int32_t rs_tiles(int32_t n) { return (n + kRsTile - 1) / kRsTile; }

template <class K>
__device__ __forceinline__ uint32_t digit_of(K k, int bit, uint32_t mask) {
    return (uint32_t)(k >> bit) & mask;
}

template <class K>
__global__ __launch_bounds__(kRsThreads) void k_rs_hist(const K *keys, int32_t n, int bit,
                                                        int nbits, int32_t n_tiles,
                                                        int32_t *counts, const int32_t *gate) {
    if (gate != nullptr && *gate == 0) return;
    __shared__ int32_t h[kRsBins];
    h[threadIdx.x] = 0;
    __syncthreads();
    const uint32_t mask = (1u << nbits) - 1;
    const int64_t base = (int64_t)blockIdx.x * kRsTile;
#pragma unroll
    for (int j = 0; j < kRsItems; j++) {
        const int64_t i = base + j * kRsThreads + threadIdx.x;
        if (i < n) atomicAdd(&h[digit_of(keys[i], bit, mask)], 1);
    }
    __syncthreads();
    counts[(int64_t)threadIdx.x * n_tiles + blockIdx.x] = h[threadIdx.x];
}

template <class K>
__global__ __launch_bounds__(kRsThreads) void k_rs_scatter(const K *keys_in,
                                                           const int32_t *vals_in, K *keys_out,
                                                           int32_t *vals_out, int32_t n, int bit,
                                                           int nbits, int32_t n_tiles,
                                                           const int32_t *offs,
                                                           const int32_t *gate) {
    if (gate != nullptr && *gate == 0) return;
    __shared__ int32_t wcnt[kRsWaves][kRsBins];   // running counts, then wave offsets
    __shared__ int32_t dbase[kRsBins];            // the tile's first slot of each digit
    __shared__ int32_t gbase[kRsBins];            // the output position of that slot
    __shared__ int32_t wsum[kRsWaves + 1];
    __shared__ K skeys[kRsTile];
    __shared__ int32_t svals[kRsTile];
    const int lane = lane_id(), w = wave_id(), tid = threadIdx.x;
#pragma unroll
    for (int ww = 0; ww < kRsWaves; ww++) wcnt[ww][tid] = 0;
    __syncthreads();
    const uint32_t mask = (1u << nbits) - 1;
    const int64_t tile0 = (int64_t)blockIdx.x * kRsTile;
    const int64_t base = tile0 + (int64_t)w * kRsWaveKeys;
    const unsigned long long below = (1ull << lane) - 1ull;
    K k[kRsItems];
    int32_t v[kRsItems];
    int32_t loc[kRsItems];
#pragma unroll
    for (int j = 0; j < kRsItems; j++) {
        const int64_t i = base + j * kWave + lane;
        k[j] = i < n ? keys_in[i] : (K)0;
        v[j] = i < n ? vals_in[i] : 0;
    }
#pragma unroll
    for (int j = 0; j < kRsItems; j++) {
        const bool valid = base + j * kWave + lane < n;
        const uint32_t d = digit_of(k[j], bit, mask);
        unsigned long long peers = __ballot(valid);
        for (int b = 0; b < nbits; b++) {
            const bool set = (d >> b) & 1u;
            const unsigned long long bal = __ballot(set);
            peers &= set ? bal : ~bal;
        }
        // peers of an invalid lane are the valid lanes that share its digit
        // bits; the lane itself takes no part below
        const int leader = peers != 0ull ? __ffsll((long long)peers) - 1 : lane;
        int32_t old = 0;
        if (valid && lane == leader) {
            old = wcnt[w][d];
            wcnt[w][d] = old + __popcll(peers);
        }
        old = __shfl(old, leader, kWave);
        loc[j] = old + __popcll(peers & below);
    }
    __syncthreads();
    // digit tid: offsets of the waves inside the tile's run of that digit
    int32_t tot = 0;
#pragma unroll
    for (int ww = 0; ww < kRsWaves; ww++) {
        const int32_t c = wcnt[ww][tid];
        wcnt[ww][tid] = tot;
        tot += c;
    }
    int32_t total;
    dbase[tid] = block_excl_scan_i32(tot, wsum, &total);
    gbase[tid] = offs[(int64_t)tid * n_tiles + blockIdx.x];
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kRsItems; j++) {
        if (base + j * kWave + lane < n) {
            const uint32_t d = digit_of(k[j], bit, mask);
            const int32_t r = dbase[d] + wcnt[w][d] + loc[j];
            skeys[r] = k[j];
            svals[r] = v[j];
        }
    }
    __syncthreads();
    const int32_t tn = (int32_t)min((int64_t)kRsTile, (int64_t)n - tile0);
    for (int32_t r = tid; r < tn; r += kRsThreads) {
        const K key = skeys[r];
        const uint32_t d = digit_of(key, bit, mask);
        const int64_t pos = (int64_t)gbase[d] + (r - dbase[d]);
        keys_out[pos] = key;
        vals_out[pos] = svals[r];
    }
}

template <class K>
__global__ void k_rs_copy(const K *ki, const int32_t *vi, K *ko, int32_t *vo, int32_t n,
                          const int32_t *gate) {
    if (gate != nullptr && *gate == 0) return;
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
        ko[i] = ki[i];
        vo[i] = vi[i];
    }
}

// ---- inclusive scan of int64 (three passes: tile sums, tile offsets, apply) ----
constexpr int kSc64Threads = 256;
constexpr int kSc64Items = 8;
constexpr int kSc64Tile = kSc64Threads * kSc64Items;

__device__ __forceinline__ long long wave_incl_scan_i64(long long x) {
    const int lane = lane_id();
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const long long y = __shfl_up(x, off, kWave);
        if (lane >= off) x += y;
    }
    return x;
}

// exclusive scan over the workgroup of one value per thread; *total = sum
__device__ __forceinline__ long long block_excl_scan_i64(long long x, long long *ws,
                                                         long long *total) {
    const int lane = lane_id(), wid = wave_id();
    constexpr int nw = kSc64Threads / kWave;
    const long long incl = wave_incl_scan_i64(x);
    if (lane == kWave - 1) ws[wid] = incl;
    __syncthreads();
    long long before = 0, all = 0;
#pragma unroll
    for (int i = 0; i < nw; i++) {
        const long long s = ws[i];
        before += i < wid ? s : 0;
        all += s;
    }
    *total = all;
    return before + incl - x;
}

__global__ __launch_bounds__(kSc64Threads) void k_sc64_sums(const int64_t *in, int32_t n,
                                                            long long *tile_sums) {
    __shared__ long long ws[kSc64Threads / kWave];
    const int64_t base = (int64_t)blockIdx.x * kSc64Tile;
    long long s = 0;
#pragma unroll
    for (int j = 0; j < kSc64Items; j++) {
        const int64_t i = base + j * kSc64Threads + threadIdx.x;
        if (i < n) s += in[i];
    }
    long long total;
    (void)block_excl_scan_i64(s, ws, &total);
    if (threadIdx.x == 0) tile_sums[blockIdx.x] = total;
}

__global__ __launch_bounds__(kSc64Threads) void k_sc64_offsets(long long *tile_sums,
                                                               int32_t n_tiles) {
    __shared__ long long ws[kSc64Threads / kWave];
    long long carry = 0;
    for (int32_t b = 0; b < n_tiles; b += kSc64Threads) {
        const int32_t i = b + threadIdx.x;
        const long long x = i < n_tiles ? tile_sums[i] : 0;
        long long total;
        const long long ex = block_excl_scan_i64(x, ws, &total);
        if (i < n_tiles) tile_sums[i] = carry + ex;
        carry += total;
        __syncthreads();
    }
}

// Each thread scans kSc64Items consecutive values: loaded through LDS so that
// the global reads and writes stay coalesced.
__global__ __launch_bounds__(kSc64Threads) void k_sc64_apply(const int64_t *in, int32_t n,
                                                             const long long *tile_offsets,
                                                             int64_t *out) {
    __shared__ long long ws[kSc64Threads / kWave];
    __shared__ long long buf[kSc64Tile + kSc64Tile / 32];
    auto slot = [](int i) { return i + i / 32; };   // padding against bank conflicts
    const int64_t base = (int64_t)blockIdx.x * kSc64Tile;
#pragma unroll
    for (int j = 0; j < kSc64Items; j++) {
        const int i = j * kSc64Threads + threadIdx.x;
        buf[slot(i)] = base + i < n ? in[base + i] : 0;
    }
    __syncthreads();
    long long x[kSc64Items];
    long long s = 0;
#pragma unroll
    for (int j = 0; j < kSc64Items; j++) {
        x[j] = buf[slot(threadIdx.x * kSc64Items + j)];
        s += x[j];
    }
    long long total;
    long long run = block_excl_scan_i64(s, ws, &total) + tile_offsets[blockIdx.x];
#pragma unroll
    for (int j = 0; j < kSc64Items; j++) {
        run += x[j];
        buf[slot(threadIdx.x * kSc64Items + j)] = run;
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kSc64Items; j++) {
        const int i = j * kSc64Threads + threadIdx.x;
        if (base + i < n) out[base + i] = buf[slot(i)];
    }
}

struct RsLayout {
    size_t keys, vals, counts, offs, ws, total;
    RsLayout(int32_t n, size_t key_bytes) {
        const size_t nt = (size_t)rs_tiles(n);
        const size_t cells = nt * kRsBins;
        size_t o = 0;
        keys = o;
        o += al256((size_t)n * key_bytes);
        vals = o;
        o += al256((size_t)n * 4);
        counts = o;
        o += al256(cells * 4);
        offs = o;
        o += al256((cells + 1) * 4);
        ws = o;
        o += al256(scan_workspace_elems((int32_t)cells) * 4);
        total = o;
    }
};

template <class K>
hipError_t sort_pairs_impl(const K *keys_in, K *keys_out, const int32_t *vals_in,
                           int32_t *vals_out, int32_t n, int begin_bit, int end_bit,
                           void *scratch, hipStream_t s, const int32_t *gate) {
    if (n <= 0) return hipSuccess;
    const int width = (int)(8 * sizeof(K));
    if (begin_bit < 0 || end_bit > width || begin_bit > end_bit) return hipErrorInvalidValue;
    const int passes = (end_bit - begin_bit + kRsBits - 1) / kRsBits;
    if (passes == 0) {
        k_rs_copy<K><<<(unsigned)std::min<int64_t>((n + 255) / 256, 4096), 256, 0, s>>>(
            keys_in, vals_in, keys_out, vals_out, n, gate);
        return hipGetLastError();
    }
    const RsLayout L(n, sizeof(K));
    char *base = reinterpret_cast<char *>(scratch);
    K *kt = reinterpret_cast<K *>(base + L.keys);
    int32_t *vt = reinterpret_cast<int32_t *>(base + L.vals);
    int32_t *counts = reinterpret_cast<int32_t *>(base + L.counts);
    int32_t *offs = reinterpret_cast<int32_t *>(base + L.offs);
    int32_t *ws = reinterpret_cast<int32_t *>(base + L.ws);
    const int32_t nt = rs_tiles(n);
    const K *ki = keys_in;
    const int32_t *vi = vals_in;
    for (int p = 0; p < passes; p++) {
        const int bit = begin_bit + p * kRsBits;
        const int nbits = std::min(kRsBits, end_bit - bit);
        // the last pass writes the outputs; earlier ones alternate so that
        // pass p writes into the buffer pass p + 1 does not write
        const bool to_out = ((passes - 1 - p) & 1) == 0;
        K *ko = to_out ? keys_out : kt;
        int32_t *vo = to_out ? vals_out : vt;
        k_rs_hist<K><<<nt, kRsThreads, 0, s>>>(ki, n, bit, nbits, nt, counts, gate);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        if ((e = launch_exclusive_scan(counts, offs, nt * kRsBins, ws, s)) != hipSuccess) return e;
        k_rs_scatter<K><<<nt, kRsThreads, 0, s>>>(ki, vi, ko, vo, n, bit, nbits, nt, offs, gate);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        ki = ko;
        vi = vo;
    }
    return hipSuccess;
}

}  // namespace

size_t sort_pairs_scratch_bytes(int32_t n, int key_bytes) {
    return RsLayout(n > 0 ? n : 0, (size_t)key_bytes).total;
}

hipError_t sort_pairs_u32(const uint32_t *keys_in, uint32_t *keys_out, const int32_t *vals_in,
                          int32_t *vals_out, int32_t n, int begin_bit, int end_bit,
                          void *scratch, hipStream_t s, const int32_t *gate) {
    return sort_pairs_impl<uint32_t>(keys_in, keys_out, vals_in, vals_out, n, begin_bit,
                                     end_bit, scratch, s, gate);
}

hipError_t sort_pairs_u64(const uint64_t *keys_in, uint64_t *keys_out, const int32_t *vals_in,
                          int32_t *vals_out, int32_t n, int begin_bit, int end_bit,
                          void *scratch, hipStream_t s, const int32_t *gate) {
    return sort_pairs_impl<uint64_t>(keys_in, keys_out, vals_in, vals_out, n, begin_bit,
                                     end_bit, scratch, s, gate);
}

size_t inclusive_scan_i64_scratch_bytes(int32_t n) {
    const int32_t nt = (n + kSc64Tile - 1) / kSc64Tile;
    return al256((size_t)(nt > 0 ? nt : 1) * 8);
}

hipError_t inclusive_scan_i64(const int64_t *in, int64_t *out, int32_t n, void *scratch,
                              hipStream_t s) {
    if (n <= 0) return hipSuccess;
    const int32_t nt = (n + kSc64Tile - 1) / kSc64Tile;
    long long *sums = reinterpret_cast<long long *>(scratch);
    k_sc64_sums<<<nt, kSc64Threads, 0, s>>>(in, n, sums);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    k_sc64_offsets<<<1, kSc64Threads, 0, s>>>(sums, nt);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    k_sc64_apply<<<nt, kSc64Threads, 0, s>>>(in, n, sums, out);
    return hipGetLastError();
}

}  // namespace pardnn
