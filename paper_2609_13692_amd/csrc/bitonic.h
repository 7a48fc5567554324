// Bitonic sort of 2^k >= kSortTile uint64 keys, ascending, on the caller's
// stream: tiles of kSortTile keys are sorted in LDS, strides of a tile or
// more run as global compare-exchange passes, the strides below a tile of
// every later stage again in LDS. Shared by the library's source files.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "common.h"

namespace mptlib {

constexpr int kSortTile = 4096;              // keys sorted in LDS per workgroup
constexpr int kSortThreads = 1024;

namespace bitonic_detail {
__device__ inline void cswap(uint64_t &a, uint64_t &b, bool up) {
    if ((a > b) == up) { const uint64_t t = a; a = b; b = t; }
}

// every stage k <= kSortTile inside one tile (direction from the global index)
static __global__ __launch_bounds__(kSortThreads) void k_sort_tile(uint64_t *keys) {
    __shared__ uint64_t t[kSortTile];
    const int64_t base = (int64_t)blockIdx.x * kSortTile;
    for (int e = threadIdx.x; e < kSortTile; e += kSortThreads) t[e] = keys[base + e];
    __syncthreads();
    for (int k = 2; k <= kSortTile; k <<= 1)
        for (int j = k >> 1; j > 0; j >>= 1) {
            for (int p = threadIdx.x; p < kSortTile / 2; p += kSortThreads) {
                // j is a power of two: the pair's lower index without a division
                const int i = ((p & ~(j - 1)) << 1) | (p & (j - 1)), l = i + j;
                cswap(t[i], t[l], ((base + i) & k) == 0);
            }
            __syncthreads();
        }
    for (int e = threadIdx.x; e < kSortTile; e += kSortThreads) keys[base + e] = t[e];
}

// one compare-exchange step of stage k with stride j >= kSortTile
static __global__ void k_sort_global(uint64_t *keys, int64_t n, int64_t k, int64_t j) {
    for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < n / 2; p += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = ((p & ~(j - 1)) << 1) | (p & (j - 1)), l = i + j;    // j: a power of two
        uint64_t a = keys[i], b = keys[l];
        cswap(a, b, (i & k) == 0);
        keys[i] = a; keys[l] = b;
    }
}

// the strides j < kSortTile of stage k > kSortTile inside one tile
static __global__ __launch_bounds__(kSortThreads) void k_sort_tile_merge(uint64_t *keys, int64_t k) {
    __shared__ uint64_t t[kSortTile];
    const int64_t base = (int64_t)blockIdx.x * kSortTile;
    for (int e = threadIdx.x; e < kSortTile; e += kSortThreads) t[e] = keys[base + e];
    __syncthreads();
    const bool up = (base & k) == 0;            // the tile lies inside one run of stage k
    for (int j = kSortTile >> 1; j > 0; j >>= 1) {
        for (int p = threadIdx.x; p < kSortTile / 2; p += kSortThreads) {
            const int i = ((p & ~(j - 1)) << 1) | (p & (j - 1)), l = i + j;
            cswap(t[i], t[l], up);
        }
        __syncthreads();
    }
    for (int e = threadIdx.x; e < kSortTile; e += kSortThreads) keys[base + e] = t[e];
}

}  // namespace bitonic_detail

// Short segments: the position of lane e's entry (key r, e < n <= 64) in
// its wave's segment, ascending by key, ties by lane: the number of lanes f
// < n with a smaller key, or an equal one and f < e. dup: some other lane
// holds an equal key. One shuffle per lane of the segment.
constexpr int kSegMax = 64;
__device__ inline int seg_rank(uint32_t r, int n, bool &dup) {
    const int e = (int)(threadIdx.x & 63u);
    int pos = 0;
    dup = false;
    for (int f = 0; f < n; ++f) {
        const uint32_t o = (uint32_t)__shfl((int)r, f, 64);
        pos += (o < r || (o == r && f < e)) ? 1 : 0;
        dup = dup || (o == r && f != e);
    }
    return pos;
}

// n must be a power of two and at least kSortTile
inline int sort_keys(uint64_t *keys, int64_t n, hipStream_t s) {
    using namespace bitonic_detail;
    const int tiles = (int)(n / kSortTile);
    k_sort_tile<<<tiles, kSortThreads, 0, s>>>(keys);
    for (int64_t k = 2 * kSortTile; k <= n; k <<= 1) {
        for (int64_t j = k >> 1; j >= kSortTile; j >>= 1)
            k_sort_global<<<grid_for(n / 2, 256, 16384), 256, 0, s>>>(keys, n, k, j);
        k_sort_tile_merge<<<tiles, kSortThreads, 0, s>>>(keys, k);
    }
    MPT_HIP_TRY(hipGetLastError());
    return MPT_OK;
}


}  // namespace mptlib
