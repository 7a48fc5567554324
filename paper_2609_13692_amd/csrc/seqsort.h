// Lexicographic sort of requests by their chunk sequences (a CSR of
// sequences: off[m+1], seqs[off[m]]): a bitonic sort of request indices with
// a comparator that reads the sequences; a proper prefix sorts first, equal
// sequences by request index. Tiles of kSeqSortTile indices are sorted in
// LDS, with the first kSeqLdsDepth chunks and the length of every request of
// the tile staged there, so that a comparison reads global memory only when
// two sequences agree on all the staged chunks. Shared by the library's
// source files.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "common.h"

namespace mptlib {

constexpr int kSeqSortTile = 1024;            // requests sorted in LDS per workgroup
constexpr int kSeqLdsDepth = 8;               // leading chunks of each request staged in LDS
constexpr int kSeqLdsStride = kSeqLdsDepth + 1;   // padded row: rows of nearby slots in distinct banks

// a < b: sequence order, a proper prefix first, equal sequences by index;
// index -1 is padding and sorts last
__device__ inline bool seq_less(int a, int b, const int64_t *off, const int32_t *seqs) {
    if (b < 0) return a >= 0;
    if (a < 0) return false;
    const int64_t la = off[a + 1] - off[a], lb = off[b + 1] - off[b];
    const int32_t *sa = seqs + off[a], *sb = seqs + off[b];
    const int64_t n = la < lb ? la : lb;
    for (int64_t j = 0; j < n; ++j)
        if (sa[j] != sb[j]) return sa[j] < sb[j];
    if (la != lb) return la < lb;
    return a < b;
}

// the same order from chunk kSeqLdsDepth on (the first kSeqLdsDepth chunks
// are equal and both sequences are longer)
__device__ inline bool seq_less_tail(int a, int b, const int64_t *off, const int32_t *seqs) {
    const int64_t la = off[a + 1] - off[a], lb = off[b + 1] - off[b];
    const int32_t *sa = seqs + off[a], *sb = seqs + off[b];
    const int64_t n = la < lb ? la : lb;
    for (int64_t j = kSeqLdsDepth; j < n; ++j)
        if (sa[j] != sb[j]) return sa[j] < sb[j];
    if (la != lb) return la < lb;
    return a < b;
}

// a tile's requests in LDS: ids (-1: padding), lengths, leading chunks
struct SeqTile {
    int32_t id[kSeqSortTile];
    int64_t len[kSeqSortTile];
    int32_t c[kSeqSortTile * kSeqLdsStride];
    int32_t t[kSeqSortTile];                  // the tile's order, as slots of the arrays above
};

__device__ inline void seq_tile_load(SeqTile &T, const int32_t *ord, int64_t base, const int64_t *off,
                                     const int32_t *seqs) {
    for (int e = threadIdx.x; e < kSeqSortTile; e += blockDim.x) {
        const int a = ord[base + e];
        T.id[e] = a;
        T.t[e] = e;
        int64_t la = 0;
        if (a >= 0) la = off[a + 1] - off[a];
        T.len[e] = la;
        const int32_t *sa = a >= 0 ? seqs + off[a] : nullptr;
#pragma unroll
        for (int j = 0; j < kSeqLdsDepth; ++j) T.c[e * kSeqLdsStride + j] = j < la ? sa[j] : 0;
    }
}

// seq_less on two slots of the tile
__device__ inline bool seq_less_slot(const SeqTile &T, int x, int y, const int64_t *off, const int32_t *seqs) {
    const int a = T.id[x], b = T.id[y];
    if (b < 0) return a >= 0;
    if (a < 0) return false;
    const int64_t la = T.len[x], lb = T.len[y];
    const int64_t n = la < lb ? la : lb;
    const int64_t nl = n < kSeqLdsDepth ? n : kSeqLdsDepth;
    for (int64_t j = 0; j < nl; ++j) {
        const int32_t u = T.c[x * kSeqLdsStride + j], v = T.c[y * kSeqLdsStride + j];
        if (u != v) return u < v;
    }
    if (n > kSeqLdsDepth) return seq_less_tail(a, b, off, seqs);
    if (la != lb) return la < lb;
    return a < b;
}

static __global__ void k_l_ord_init(int m, int64_t mpad, int32_t *ord) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < mpad; i += (int64_t)gridDim.x * blockDim.x)
        ord[i] = i < m ? (int32_t)i : -1;
}

// all stages with k <= kSeqSortTile inside one tile of request indices
static __global__ __launch_bounds__(256) void k_l_seq_sort_tile(int32_t *ord, const int64_t *off, const int32_t *seqs) {
    __shared__ SeqTile T;
    const int64_t base = (int64_t)blockIdx.x * kSeqSortTile;
    seq_tile_load(T, ord, base, off, seqs);
    __syncthreads();
    for (int k = 2; k <= kSeqSortTile; k <<= 1)
        for (int j = k >> 1; j > 0; j >>= 1) {
            for (int p = threadIdx.x; p < kSeqSortTile / 2; p += blockDim.x) {
                const int i = ((p & ~(j - 1)) << 1) | (p & (j - 1)), l = i + j;    // j: a power of two
                const bool up = ((base + i) & k) == 0;
                const int x = T.t[i], y = T.t[l];
                if (seq_less_slot(T, y, x, off, seqs) == up) { T.t[i] = y; T.t[l] = x; }
            }
            __syncthreads();
        }
    for (int e = threadIdx.x; e < kSeqSortTile; e += blockDim.x) ord[base + e] = T.id[T.t[e]];
}

static __global__ void k_l_seq_sort_global(int32_t *ord, int64_t n, int64_t k, int64_t j, const int64_t *off,
                                    const int32_t *seqs) {
    for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < n / 2; p += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = ((p & ~(j - 1)) << 1) | (p & (j - 1)), l = i + j;    // j: a power of two
        const bool up = (i & k) == 0;
        const int a = ord[i], b = ord[l];
        if (seq_less(b, a, off, seqs) == up) { ord[i] = b; ord[l] = a; }
    }
}

static __global__ __launch_bounds__(256) void k_l_seq_sort_tile_merge(int32_t *ord, int64_t k, const int64_t *off,
                                                               const int32_t *seqs) {
    __shared__ SeqTile T;
    const int64_t base = (int64_t)blockIdx.x * kSeqSortTile;
    seq_tile_load(T, ord, base, off, seqs);
    __syncthreads();
    const bool up = (base & k) == 0;
    for (int j = kSeqSortTile >> 1; j > 0; j >>= 1) {
        for (int p = threadIdx.x; p < kSeqSortTile / 2; p += blockDim.x) {
            const int i = ((p & ~(j - 1)) << 1) | (p & (j - 1)), l = i + j;    // j: a power of two
            const int x = T.t[i], y = T.t[l];
            if (seq_less_slot(T, y, x, off, seqs) == up) { T.t[i] = y; T.t[l] = x; }
        }
        __syncthreads();
    }
    for (int e = threadIdx.x; e < kSeqSortTile; e += blockDim.x) ord[base + e] = T.id[T.t[e]];
}

// ord[0 .. n) gets the request ids 0 .. m-1 in order, then -1 (padding);
// n is a power of two, at least kSeqSortTile
inline int sort_requests(int32_t *ord, int m, int64_t n, const int64_t *off, const int32_t *seqs, hipStream_t s) {
    const int tiles = (int)(n / kSeqSortTile);
    k_l_ord_init<<<grid_for(n, 256), 256, 0, s>>>(m, n, ord);
    k_l_seq_sort_tile<<<tiles, 256, 0, s>>>(ord, off, seqs);
    for (int64_t k = 2 * kSeqSortTile; k <= n; k <<= 1) {
        for (int64_t j = k >> 1; j >= kSeqSortTile; j >>= 1)
            k_l_seq_sort_global<<<grid_for(n / 2, 256, 16384), 256, 0, s>>>(ord, n, k, j, off, seqs);
        k_l_seq_sort_tile_merge<<<tiles, 256, 0, s>>>(ord, k, off, seqs);
    }
    MPT_HIP_TRY(hipGetLastError());
    return MPT_OK;
}

}  // namespace mptlib
