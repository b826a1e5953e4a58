// Sums of a vector over the set bits of packed 0/1 rows through "nibble
// tables" in LDS: for 4 consecutive entries of the vector, the sums over all
// 16 subsets, so that the sum over the set bits of a 64-bit word is 16 table
// reads (Sec. 3.5's least squares applies the sampled masks and their
// transpose to vectors this way, straight from the bits).
#pragma once

#include "common.h"

namespace gnnshap {

constexpr int64_t kTabWords = 16;    // nibble tables per workgroup: 16 words (32 KiB of LDS)

// Nibble tables: for 64 consecutive entries v[0..63] of a vector, table k
// (k = 0..15) holds at index n the sum of v[4k + i] over the set bits i of n,
// so that the sum of v over the set bits of a 64-bit word is the sum of 16
// table reads.  One table is 16 fp64 entries, 128 bytes: its entries fall in
// distinct LDS banks, so 64 lanes reading one table never conflict.  The
// tables of a workgroup are one static LDS array, word w's 16 tables at
// byte 2048 w.
//
// ntab tables of v (4 entries each) into tab, consecutive threads on
// consecutive entries, so the writes of a wavefront cover 512 contiguous
// bytes (no two lanes in one bank).  Entry n of table q is
// ((v[4q] [n & 1] + v[4q + 1] [n & 2]) + v[4q + 2] [n & 4]) + v[4q + 3] [n & 8],
// an absent term adding 0.0 (exact).
__device__ __forceinline__ void build_tables(const double* __restrict__ v, int64_t ntab, double* tab) {
  for (int64_t e = threadIdx.x; e < ntab * 16; e += blockDim.x) {
    const double* v4 = v + (e >> 4) * 4;
    const int n = static_cast<int>(e & 15);
    const double a0 = (n & 1) ? v4[0] : 0.0;
    const double a1 = (n & 2) ? v4[1] : 0.0;
    const double a2 = (n & 4) ? v4[2] : 0.0;
    const double a3 = (n & 8) ? v4[3] : 0.0;
    tab[e] = ((a0 + a1) + a2) + a3;
  }
}

// acc[0..3] += sum over the set bits b of word of v[b], from the word's 16
// tables at byte 2048 W of `tabs` (W a constant, so that the table offsets
// are immediates of the LDS reads).  Each 32-bit half is masked into two
// words whose bytes hold 8 x a nibble (the byte offset of the entry in its
// table): one extract per nibble gives the LDS address.  Table t adds into
// acc[t & 3], tables in ascending order.
template <int W>
__device__ __forceinline__ void nibble_dot(uint64_t word, const char* tabs, double (&acc)[4]) {
  constexpr uint32_t kM = 0x78787878u;
  const uint32_t lo = static_cast<uint32_t>(word), hi = static_cast<uint32_t>(word >> 32);
  const uint32_t q[4] = {(lo << 3) & kM, (lo >> 1) & kM, (hi << 3) & kM, (hi >> 1) & kM};
#pragma unroll
  for (int half = 0; half < 2; ++half)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int odd = 0; odd < 2; ++odd) {
        const int t = 8 * half + 2 * j + odd;
        const uint32_t off = __builtin_amdgcn_ubfe(q[2 * half + odd], 8 * j, 8);
        acc[t & 3] += *reinterpret_cast<const double*>(tabs + (W * 2048 + t * 128) + off);
      }
}

// acc[0..3] += the products of n <= NW words (word w at src[w * stride]) with
// the tables of consecutive 64-entry groups; the next word's load is issued
// before the current word's table reads.
template <int NW, int W = 0>
__device__ __forceinline__ void nibble_dots(const uint64_t* __restrict__ src, int64_t stride, int n, uint64_t next,
                                            const char* tabs, double (&acc)[4]) {
  if constexpr (W < NW) {
    if (W >= n) return;
    const uint64_t word = next;
    if (W + 1 < n) next = src[(W + 1) * stride];
    nibble_dot<W>(word, tabs, acc);
    nibble_dots<NW, W + 1>(src, stride, n, next, tabs, acc);
  }
}

// build_tables for a vector of n valid entries (entries from n on read as 0).
__device__ __forceinline__ void build_tables_bounded(const double* __restrict__ v, int64_t n, int64_t ntab,
                                                     double* tab) {
  for (int64_t e = threadIdx.x; e < ntab * 16; e += blockDim.x) {
    const int64_t i0 = (e >> 4) * 4;
    const int sub = static_cast<int>(e & 15);
    const double a0 = ((sub & 1) && i0 < n) ? v[i0] : 0.0;
    const double a1 = ((sub & 2) && i0 + 1 < n) ? v[i0 + 1] : 0.0;
    const double a2 = ((sub & 4) && i0 + 2 < n) ? v[i0 + 2] : 0.0;
    const double a3 = ((sub & 8) && i0 + 3 < n) ? v[i0 + 3] : 0.0;
    tab[e] = ((a0 + a1) + a2) + a3;
  }
}

}  // namespace gnnshap
