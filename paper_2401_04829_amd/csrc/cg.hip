// Matrix-free conjugate gradients for the projected Kernel-SHAP normal
// equations (Sec. 3.5 of the GNNShap paper: above 5000 players the regression
// is fitted iteratively rather than by a direct solve).
//
// Unknown psi in 1-perp, phi = Delta/M + psi.  With R the random
// representative rows (each stands for itself and its complement) and P the
// centring projector, the operator on 1-perp is
//     A v = alpha v + 2 w_r P R^T (R v),
// alpha collecting the enumerated classes (their projected Gram is a multiple
// of P).  No Gram matrix is formed: every iteration applies R and R^T to the
// residual straight from the packed bits.
//
// The recurrences are those of Chronopoulos and Gear's conjugate gradients
// (SIAM J. Sci. Stat. Comput. 1989), which apply A to the residual r and
// carry s = A p along: with w = A r, gamma = r.r and delta = r.w,
//     beta = gamma / gamma_prev, a = gamma / (delta - beta gamma / a_prev),
//     p = r + beta p, s = w + beta s, x += a p, r -= a s.
// Every vector a pass reads was finished by an earlier kernel.  Each
// workgroup turns its slice of that vector into nibble tables in LDS (sums of
// the vector over every subset of 4 consecutive entries); each lane then
// loads its own mask word with ordinary vector loads and adds one table entry
// per 4 bits (a bit extract, an address and an fp64 add per nibble, instead
// of a multiply-add per bit).  delta needs no extra reduction:
// r.A r = alpha |r|^2 + 2 w_r |R r|^2 for r in 1-perp.
//
// Rows of small coalitions are mostly zero bits: the random rows whose size
// is at most M / kSparseDiv (the first ones: the plan orders random classes
// by ascending size), in whole blocks of 64 rows, are kept as lists of their
// players instead (sparse rows), built once per solve from the bits, row by
// row and player by player (both in ascending order).  In pass A a group of
// L lanes sums one row's list (each lane at most about four entries, then a
// fixed butterfly over the group), L fixed per block of 64 rows from the
// block's largest row, so a wavefront takes 64 / L rows at once; in pass B
// groups of lanes sized from the mean list length sum the players' lists.
//
// Per iteration t:
//   pass A   stopping test on gamma_t; partial products R r of the bit rows
//            over player chunks (lane = row, the rows' words in row blocks)
//            and, in workgroups of their own in the same launch, u = R r of
//            the sparse rows (a wavefront sums r over a row's players);
//   rows     u of the bit rows (the sum of their chunks); partial |u|^2, |m|.u;
//   pass B   partial products R^T u of the bit rows over row chunks (lane =
//            player, words of the bit-transposed rows) and, in workgroups of
//            their own, the sparse rows' R_s^T u (a wavefront per player);
//   update   w = alpha r + 2 w_r (R^T u - mean), the scalars, the vector steps
//            and the partial sums of the new gamma.
// Vectors and every sum are fp64; partial sums are reduced in a fixed order,
// so repeated solves give the same bits.  The iteration stops when
// |r| <= kTol |r_0| or after kMaxIt iterations; the host queues iterations in
// chunks and checks a flag the device writes to mapped host memory, so at
// most one chunk runs idle.
#include <algorithm>
#include <atomic>
#include <vector>

#include "cg.h"
#include "nibble.h"

namespace {

using gnnshap::build_tables;
using gnnshap::nibble_dots;

// Relative residual at which the iteration stops.  On the Reddit-shaped
// targets (10,793-30,000 players, 100,000 coalitions) phi then differs from
// a solve to 1e-10 by at most 4.6e-6 of max|phi| (1e-7: 4.9e-7; 1e-8:
// 6e-8), far inside the 1e-3 bar that the solution is held to, at 3/4 of
// the iterations that 1e-8 takes.
constexpr double kTol = 1e-6;
constexpr int64_t kMaxIt = 4000;
constexpr int64_t kChunk = 8;        // iterations queued between stopping checks
constexpr int kWaves = 16;           // waves per workgroup of both passes
constexpr int kTabA = 32;            // pass A: words of r's tables per workgroup (64 KiB of LDS)
constexpr int kTabB = 32;            // pass B: row blocks of u's tables per workgroup
constexpr int kPerWaveGroup = 2;     // row blocks (pass A) and player words (pass B) per wavefront
                                     // in a group of several systems; one for a system alone
constexpr int64_t kFill = 4096;      // (row block, chunk) pairs of a pass per system, at least
constexpr int64_t kSparseDiv = 128;   // sparse rows: coalition size at most M / kSparseDiv

struct Args {
  const uint64_t* blocked;   // the bit rows in row blocks (pass A)
  const uint64_t* T;         // the bit rows transposed (pass B)
  const int32_t* sz;
  int64_t M, wpr, kr, nrb, npc, pwords, nrc, rbc, nbu, nbc;
  int64_t rs, rbd0, nsa, nsb, nrcd, nxa, nxb, nsi;
  int32_t pw;                // row blocks / player words per wavefront of the two passes (their grids)
  int32_t lgb;     // pass B: log2 of the lanes summing one player's list
  const int64_t* sitem;
  const int64_t* csr_ptr;
  const int32_t* csr_idx;
  const int64_t* csc_ptr;
  const int32_t* csc_row;
  double* qs;
  double alpha, wr2, tol2;
  int64_t maxit;
  int32_t has_random;
  double* x;
  double* r;       // wpr * 64 (zero beyond M)
  double* p;
  double* s;
  double* upart;
  double* u;       // nrb * 64 (zero beyond kr)
  double* qpart;
  double* uu;
  double* usp;     // 2 x nsa: pass A's sparse-row partials
  double* rr;      // 3 x nbc
  double* hist;    // step length of even and odd iterations
  gnnshap::CgState* st;
  int32_t* host_flag;  // mapped host memory: [0] done, [1] iterations
};

// The members of one launch of a pass: member m owns workgroups
// [blk[m], blk[m + 1]) of the flat grid and runs iteration t[m].
struct GroupArgs {
  Args a[gnnshap::kCgGroupMax];
  int64_t t[gnnshap::kCgGroupMax];
  uint32_t blk[gnnshap::kCgGroupMax + 1];
  int32_t n;
};

// The member of this workgroup and the workgroup's index within it.
__device__ __forceinline__ int member_of(const GroupArgs& g, int64_t& bid) {
  const uint32_t b = blockIdx.x;
  int m = 0;
  while (m + 1 < g.n && b >= g.blk[m + 1]) ++m;
  bid = static_cast<int64_t>(b - g.blk[m]);
  return m;
}

__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  return v;
}

// Sum of a block's values v over its threads (blockDim.x a multiple of 64,
// at most 1024); the result is returned to every thread.
__device__ __forceinline__ double block_sum_d(double v, double* red) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, nw = blockDim.x >> 6;
  v = wave_sum_d(v);
  __syncthreads();
  if (lane == 0) red[wv] = v;
  __syncthreads();
  double s = 0.0;
  for (int i = 0; i < nw; ++i) s += red[i];
  return s;
}

// Sum of n values by one whole wave in a fixed order: lane l adds entries
// l, l + 64, ..., then a fixed butterfly; every wave gets the same bits.
__device__ __forceinline__ double wave_fixed_sum(const double* __restrict__ a, int64_t n, int64_t stride = 1) {
  double s = 0.0;
  for (int64_t i = threadIdx.x & 63; i < n; i += 64) s += a[i * stride];
  return wave_sum_d(s);
}

// r = dv - mean(dv) (zero beyond M), x = p = s = 0, partial gamma_0; u zero
// beyond kr; sizes of the random rows.  Grid: nbc workgroups of 256.
__global__ void __launch_bounds__(256) k_cg_init(Args a, const double* __restrict__ dv,
                                                 const double* __restrict__ bsum, int64_t nb,
                                                 const gnnshap_class* __restrict__ cls, int64_t ncls, int64_t rb0,
                                                 int32_t* sz) {
  __shared__ double red[4];
  __shared__ double mean;
  if (threadIdx.x == 0) {
    double sm = 0.0;
    for (int64_t i = 0; i < nb; ++i) sm += bsum[i];
    mean = sm / static_cast<double>(a.M);
  }
  __syncthreads();
  const int64_t j = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  double r2 = 0.0;
  if (j < a.wpr * 64) {
    const double rj = j < a.M ? dv[j] - mean : 0.0;
    a.r[j] = rj;
    r2 = rj * rj;
    if (j < a.M) {
      a.x[j] = 0.0;
      a.p[j] = 0.0;
      a.s[j] = 0.0;
    }
  }
  const double sb = block_sum_d(r2, red);
  if (threadIdx.x == 0) a.rr[blockIdx.x] = sb;   // gamma_0: slot 0
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    a.st->done = 0;
    a.st->iters = 0;
    a.st->status = 0;
  }
  const int64_t stride = static_cast<int64_t>(gridDim.x) * 256;
  for (int64_t b = a.kr + j; b < a.nrb * 64; b += stride) a.u[b] = 0.0;
  // row sizes: class of row rb0 + b by binary search over row_begin
  for (int64_t b = j; b < a.kr; b += stride) {
    const int64_t row = rb0 + b;
    int64_t lo = 0, hi = ncls - 1;
    while (lo < hi) {
      const int64_t mid = (lo + hi + 1) >> 1;
      if (cls[mid].row_begin <= row) lo = mid; else hi = mid - 1;
    }
    sz[b] = cls[lo].size;
  }
}

// Lanes per sparse row (as log2) for a block of 64 rows whose largest row
// has c players: the power of two that gives each lane at most about four
// entries, at most 64.  Host and device use the same rule.
__host__ __device__ __forceinline__ int sparse_lanes_log2(int64_t c) {
  const int64_t need = (c + 3) / 4;
  int lg = 0;
  while (lg < 6 && (int64_t(1) << lg) < need) ++lg;
  return lg;
}

// Stopping test of iteration t, taken identically by every wave of pass A
// from the partial sums of gamma_t; `writer` records the stop.
__device__ __forceinline__ bool cg_stop(const Args& a, int64_t t, bool writer) {
  const double g = wave_fixed_sum(a.rr + (t % 3) * a.nbc, a.nbc);
  const double g0 = t == 0 ? g : a.st->rr0;
  const bool bad = !(g == g) || g > 1e300;
  const bool conv = !bad && g <= a.tol2 * g0;
  if (conv || bad || t >= a.maxit) {
    if (writer) {
      a.st->done = 1;
      a.st->iters = static_cast<int32_t>(t);
      a.st->status = conv ? 0 : (bad ? 2 : 1);
      __hip_atomic_store(a.host_flag + 1, static_cast<int32_t>(t), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
      __hip_atomic_store(a.host_flag, 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
    }
    return true;
  }
  if (t == 0 && writer) a.st->rr0 = g;
  return false;
}

// Sum of the entries of v selected by n indices, by one wavefront: lane l
// takes indices l, l + 64, ... four at a time (their loads issued together),
// then a fixed butterfly; every lane gets the same bits.
__device__ __forceinline__ double wave_gather_sum(const int32_t* __restrict__ idx, int64_t n,
                                                  const double* __restrict__ v) {
  const int lane = threadIdx.x & 63;
  double s4[4] = {0.0, 0.0, 0.0, 0.0};
  int64_t e = lane;
  for (; e + 192 < n; e += 256) {
    const int32_t j0 = idx[e], j1 = idx[e + 64], j2 = idx[e + 128], j3 = idx[e + 192];
    s4[0] += v[j0];
    s4[1] += v[j1];
    s4[2] += v[j2];
    s4[3] += v[j3];
  }
  for (int q = 0; e < n; e += 64, ++q) s4[q] += v[idx[e]];
  return wave_sum_d((s4[0] + s4[1]) + (s4[2] + s4[3]));
}

// Pass A.  Workgroup y * nxa + x (y < npc): upart[y, b] = sum over the words
// of player chunk y of the bits of bit row b times r; the workgroup builds
// the chunk's nibble tables of r in LDS (r is padded with zeros to whole
// words), then each wave takes PW blocks of 64 rows (lane = row),
// reads their row-blocked words, 512 contiguous bytes per word, and sums
// table entries.  Workgroup
// nxa * npc + x (x < nsa): the sparse rows x * kWaves + wave, + nsa * kWaves,
// ...: u_b = sum of r over the row's players, with the workgroup's partial
// |u|^2 and |m|.u in uu[2 x], uu[2 x + 1].  Both kinds take the stopping
// test first.
template <int PW>
__global__ void __launch_bounds__(kWaves * 64) __attribute__((amdgpu_waves_per_eu(8))) k_cg_pass_a(GroupArgs g) {
  __shared__ double tab[kTabA * 256];   // the sparse rows' workgroups: kWaves block sums
  int64_t bid;
  const int m = member_of(g, bid);
  const Args& a = g.a[m];
  const int64_t t = g.t[m];
  if (a.st->done) return;
  const uint64_t* __restrict__ blocked = a.blocked;
  const double* __restrict__ r = a.r;
  double* __restrict__ upart = a.upart;
  // one flat grid per member: nxa x npc bit-row workgroups, then nsa sparse-row ones
  const int64_t pc = bid < a.nxa * a.npc ? bid / a.nxa : a.npc;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const bool writer = bid == 0 && threadIdx.x == 0;
  if (pc == a.npc) {                  // sparse rows
    if (cg_stop(a, t, false)) return;
    const int64_t x = bid - a.nxa * a.npc;
    double uu = 0.0, su = 0.0;
    for (int64_t it = x * kWaves + wave; it < a.nsi; it += a.nsa * kWaves) {
      const int64_t info = a.sitem[it];
      const int lg = static_cast<int>(info & 0xff);
      const int64_t b = (info >> 8) + (lane >> lg);   // this lane group's row
      const int64_t e0 = a.csr_ptr[b], e1 = a.csr_ptr[b + 1];
      double v;
      if (lg == 6) {
        v = wave_gather_sum(a.csr_idx + e0, e1 - e0, r);
      } else {
        // at most four entries per lane (the block's rows have at most 4 L
        // players), their loads issued together
        const int L = 1 << lg;
        const int64_t e = e0 + (lane & (L - 1));
        const double v0 = e < e1 ? r[a.csr_idx[e]] : 0.0;
        const double v1 = e + L < e1 ? r[a.csr_idx[e + L]] : 0.0;
        const double v2 = e + 2 * L < e1 ? r[a.csr_idx[e + 2 * L]] : 0.0;
        const double v3 = e + 3 * L < e1 ? r[a.csr_idx[e + 3 * L]] : 0.0;
        v = (v0 + v1) + (v2 + v3);
        for (int off = L >> 1; off > 0; off >>= 1) v += __shfl_xor(v, off);
      }
      if ((lane & ((1 << lg) - 1)) == 0) {
        a.u[b] = v;
        uu += v * v;
        su += static_cast<double>(a.sz[b]) * v;
      }
    }
    const double s1 = block_sum_d(uu, tab);
    const double s2 = block_sum_d(su, tab);
    if (threadIdx.x == 0) {
      a.usp[2 * x] = s1;
      a.usp[2 * x + 1] = s2;
    }
    return;
  }
  // the wavefront's row blocks: rb, rb + kWaves, ... (PW of them)
  const int64_t rb = a.rbd0 + (bid % a.nxa) * (kWaves * PW) + wave;
  const int64_t w0 = pc * a.pwords;
  const int64_t w1 = w0 + a.pwords < a.wpr ? w0 + a.pwords : a.wpr;
  const int64_t nw = w1 - w0;
  // the tables do not depend on the stopping test: built first, so that the
  // test's reads overlap them
  build_tables(r + w0 * 64, nw * 16, tab);
  if (cg_stop(a, t, writer)) return;   // the same outcome in every wave
  __syncthreads();
#pragma unroll 1
  for (int q = 0; q < PW; ++q) {
    const int64_t rq = rb + q * kWaves;
    if (rq >= a.nrb) break;
    const uint64_t* src = blocked + (rq * a.wpr + w0) * 64 + lane;
    double acc[4] = {0.0, 0.0, 0.0, 0.0};
    nibble_dots<kTabA>(src, 64, static_cast<int>(nw), src[0], reinterpret_cast<const char*>(tab), acc);
    const int64_t row = rq * 64 + lane;
    if (row < a.kr) upart[pc * a.kr + row] = (acc[0] + acc[1]) + (acc[2] + acc[3]);
  }
}

// v0 + x[0] + x[stride] + ... + x[(n - 1) stride], added in that order, with
// eight loads in flight ahead of their adds.
__device__ __forceinline__ double chunk_sum(const double* __restrict__ x, int64_t stride, int64_t n,
                                            double v0 = 0.0) {
  double v = v0;
  int64_t c = 0;
  for (; c + 8 <= n; c += 8) {
    double t[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) t[q] = x[(c + q) * stride];
#pragma unroll
    for (int q = 0; q < 8; ++q) v += t[q];
  }
  for (; c < n; ++c) v += x[c * stride];
  return v;
}

// u of the bit rows (the sum of their pass-A chunks, one lane per row) with
// partial |u|^2 and |m|.u in uu[2 (1 + x)], uu[2 (1 + x) + 1]; the last
// workgroup adds pass A's sparse-row partials into uu[0], uu[1] (fixed order).
__global__ void __launch_bounds__(256) k_cg_rows(GroupArgs g) {
  __shared__ double red[4];
  int64_t bid;
  const Args& a = g.a[member_of(g, bid)];
  if (a.st->done) return;
  if (bid == a.nbu - 1) {
    const int wv = threadIdx.x >> 6;
    if (wv < 2) {
      const double v = a.nsa > 0 ? wave_fixed_sum(a.usp + wv, a.nsa, 2) : 0.0;
      if ((threadIdx.x & 63) == 0) a.uu[wv] = v;
    }
    return;
  }
  const int64_t b = a.rs + bid * 256 + threadIdx.x;
  double uu = 0.0, su = 0.0;
  if (b < a.kr) {
    const double v = chunk_sum(a.upart + b, a.kr, a.npc);
    a.u[b] = v;
    uu = v * v;
    su = static_cast<double>(a.sz[b]) * v;
  }
  const double s1 = block_sum_d(uu, red);
  const double s2 = block_sum_d(su, red);
  if (threadIdx.x == 0) {
    a.uu[2 * (1 + bid)] = s1;
    a.uu[2 * (1 + bid) + 1] = s2;
  }
}

// Pass B.  Workgroup c * nxb + x (c < nrcd): qpart[c, j] = sum over the row
// blocks of chunk c of the bits of player j times u; the workgroup builds
// the chunk's nibble tables of u in LDS (u is padded with zeros to whole row
// blocks), then each wave takes PW words of 64 players (lane =
// player), reads the bit-transposed words T[rb, j] and sums table entries.  Workgroup
// nxb * nrcd + x (x < nsb): groups of 64 / L players (x * kWaves + wave, +
// nsb * kWaves, ...): qs[j] = sum of u over the sparse rows holding player j.
template <int PW>
__global__ void __launch_bounds__(kWaves * 64) __attribute__((amdgpu_waves_per_eu(8))) k_cg_pass_b(GroupArgs g) {
  __shared__ double tab[kTabB * 256];
  int64_t bid;
  const Args& a = g.a[member_of(g, bid)];
  if (a.st->done) return;
  const uint64_t* __restrict__ T = a.T;
  const double* __restrict__ u = a.u;
  double* __restrict__ qpart = a.qpart;
  // one flat grid per member: nxb x nrcd bit-row workgroups, then nsb sparse-row ones
  const int64_t c = bid < a.nxb * a.nrcd ? bid / a.nxb : a.nrcd;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (c == a.nrcd) {                  // sparse rows: 64 / L players per wavefront
    const int64_t x = bid - a.nxb * a.nrcd;
    const int lg = a.lgb, L = 1 << lg;
    const int64_t nit = (a.M + (64 >> lg) - 1) >> (6 - lg);
    for (int64_t it = x * kWaves + wave; it < nit; it += a.nsb * kWaves) {
      const int64_t j = (it << (6 - lg)) + (lane >> lg);
      double v;
      if (lg == 6) {
        const int64_t e0 = a.csc_ptr[j];
        v = wave_gather_sum(a.csc_row + e0, a.csc_ptr[j + 1] - e0, u);
      } else {
        const bool ok = j < a.M;
        const int64_t e1 = ok ? a.csc_ptr[j + 1] : 0;
        double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0;
        for (int64_t e = (ok ? a.csc_ptr[j] : 0) + (lane & (L - 1)); e < e1; e += 4 * L) {
          s0 += u[a.csc_row[e]];
          if (e + L < e1) s1 += u[a.csc_row[e + L]];
          if (e + 2 * L < e1) s2 += u[a.csc_row[e + 2 * L]];
          if (e + 3 * L < e1) s3 += u[a.csc_row[e + 3 * L]];
        }
        v = (s0 + s1) + (s2 + s3);
        for (int off = L >> 1; off > 0; off >>= 1) v += __shfl_xor(v, off);
      }
      if ((lane & (L - 1)) == 0 && j < a.M) a.qs[j] = v;
    }
    return;
  }
  // the wavefront's player words: gw, gw + kWaves, ... (PW of them)
  const int64_t gw = (bid % a.nxb) * (kWaves * PW) + wave;
  const int64_t b0 = a.rbd0 + c * a.rbc;
  const int64_t b1 = b0 + a.rbc < a.nrb ? b0 + a.rbc : a.nrb;
  const int64_t nb = b1 - b0;
  build_tables(u + b0 * 64, nb * 16, tab);
  __syncthreads();
#pragma unroll 1
  for (int q = 0; q < PW; ++q) {
    const int64_t gq = gw + q * kWaves;
    if (gq >= a.wpr) break;
    const int64_t j = gq * 64 + lane;
    const bool valid = j < a.M;
    const uint64_t* col = T + b0 * a.M + (valid ? j : 0);
    double acc[4] = {0.0, 0.0, 0.0, 0.0};
    // a lane beyond M reads player 0's words and discards its sums
    nibble_dots<kTabB>(col, a.M, static_cast<int>(nb), col[0], reinterpret_cast<const char*>(tab), acc);
    if (valid) qpart[c * a.M + j] = (acc[0] + acc[1]) + (acc[2] + acc[3]);
  }
}

// ---- the sparse rows' lists, built once per solve ------------------------------------------

// Exclusive prefix sums of n values by one workgroup of 1024 threads (thread t
// takes a contiguous run), v[i] -> out[i], total -> out[n].
template <class T>
__device__ void block_scan_i64(const T* __restrict__ v, int64_t n, int64_t* __restrict__ out) {
  __shared__ int64_t part[1024];
  const int t = threadIdx.x;
  const int64_t per = (n + 1023) / 1024;
  const int64_t i0 = t * per, i1 = i0 + per < n ? i0 + per : n;
  int64_t s = 0;
  for (int64_t i = i0; i < i1; ++i) s += v[i];
  part[t] = s;
  __syncthreads();
  if (t == 0) {
    int64_t run = 0;
    for (int i = 0; i < 1024; ++i) {
      const int64_t x = part[i];
      part[i] = run;
      run += x;
    }
    out[n] = run;
  }
  __syncthreads();
  int64_t run = part[t];
  for (int64_t i = i0; i < i1; ++i) {
    const int64_t x = v[i];
    out[i] = run;
    run += x;
  }
}

// Row-major lists: csr_ptr = exclusive prefix sums of the sparse rows' sizes.
__global__ void __launch_bounds__(1024) k_cg_csr_ptr(const int32_t* __restrict__ sz, int64_t rs,
                                                     int64_t* __restrict__ ptr, int64_t* __restrict__ sitem) {
  block_scan_i64(sz, rs, ptr);
  // pass A's work items: block q (rows 64 q .. 64 q + 63, sizes ascending)
  // gives 2^lg items of 64 / 2^lg rows each, lg from its largest row
  // (at most 1024 blocks: thread q owns block q; an inclusive scan of the
  // item counts in LDS, Hillis-Steele)
  __shared__ int64_t cnt[2][1024];
  const int64_t nblk = rs / 64;
  const int q = threadIdx.x;
  const int lg = q < nblk ? sparse_lanes_log2(sz[64 * q + 63]) : 0;
  cnt[0][q] = q < nblk ? (int64_t(1) << lg) : 0;
  __syncthreads();
  int cur = 0;
  for (int off = 1; off < 1024; off <<= 1) {
    cnt[cur ^ 1][q] = cnt[cur][q] + (q >= off ? cnt[cur][q - off] : 0);
    cur ^= 1;
    __syncthreads();
  }
  if (q < nblk) {
    const int64_t first = cnt[cur][q] - (int64_t(1) << lg);
    const int64_t rows = int64_t(64) >> lg;
    for (int64_t g = 0; g < (int64_t(1) << lg); ++g) sitem[first + g] = ((int64_t(64) * q + g * rows) << 8) | lg;
  }
}

// The lists are built in kSeg segments at once: of the player words for the
// row lists, of the row blocks for the player lists.  A count pass gives each
// (row or player, segment) its number of entries, so the fill pass of a
// segment starts at the list's start plus the counts of the segments before
// it; every list comes out in ascending order.
constexpr int kSeg = 8;

// Row-major lists, counts: wavefront (g, s) reads the words of segment s of its
// 64 rows from the row-blocked copy (lane = row): cnt[s][b].
__global__ void __launch_bounds__(64) k_cg_csr_count(const uint64_t* __restrict__ blocked, int64_t wpr, int64_t rs,
                                                     int32_t* __restrict__ cnt) {
  const int64_t g = blockIdx.x;
  const int sg = blockIdx.y;
  const int64_t b = g * 64 + threadIdx.x;
  if (b >= rs) return;
  const int64_t w0 = wpr * sg / kSeg, w1 = wpr * (sg + 1) / kSeg;
  const uint64_t* src = blocked + g * wpr * 64 + threadIdx.x;
  int c = 0;
  for (int64_t w = w0; w < w1; ++w) c += __popcll(src[w * 64]);
  cnt[sg * rs + b] = c;
}

// Row-major lists, fill: the players of segment s of row b in order.
__global__ void __launch_bounds__(64) k_cg_csr_fill(const uint64_t* __restrict__ blocked, int64_t wpr, int64_t rs,
                                                    const int64_t* __restrict__ ptr, const int32_t* __restrict__ cnt,
                                                    int64_t nnz, int32_t* __restrict__ idx) {
  const int64_t g = blockIdx.x;
  const int sg = blockIdx.y;
  const int64_t b = g * 64 + threadIdx.x;
  if (b >= rs) return;
  int64_t pos = ptr[b];
  for (int q = 0; q < sg; ++q) pos += cnt[q * rs + b];
  const int64_t end = ptr[b + 1] < nnz ? ptr[b + 1] : nnz;
  const int64_t w0 = wpr * sg / kSeg, w1 = wpr * (sg + 1) / kSeg;
  const uint64_t* src = blocked + g * wpr * 64 + threadIdx.x;
  for (int64_t w = w0; w < w1; ++w) {
    uint64_t word = src[w * 64];
    while (word && pos < end) {
      idx[pos++] = static_cast<int32_t>(w * 64 + __builtin_ctzll(word));
      word &= word - 1;
    }
  }
}

// Player-major lists, counts: cnt[s][j] = the sparse rows of segment s (row
// blocks nrb_s s / kSeg .. of the bit-transposed rows T[rb, j]) holding j.
__global__ void __launch_bounds__(256) k_cg_csc_count(const uint64_t* __restrict__ T, int64_t M, int64_t nrb_s,
                                                      int32_t* __restrict__ cnt) {
  const int64_t j = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const int sg = blockIdx.y;
  if (j >= M) return;
  const int64_t r0 = nrb_s * sg / kSeg, r1 = nrb_s * (sg + 1) / kSeg;
  int c = 0;
  for (int64_t rb = r0; rb < r1; ++rb) c += __popcll(T[rb * M + j]);
  cnt[sg * M + j] = c;
}

// ptr[j] = total of player j's segment counts (fixed order), then the
// exclusive prefix sums over j in place (ptr[M] = the total).
__global__ void __launch_bounds__(256) k_cg_csc_total(const int32_t* __restrict__ cnt, int64_t M,
                                                      int64_t* __restrict__ ptr) {
  const int64_t j = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (j >= M) return;
  int64_t v = 0;
#pragma unroll
  for (int q = 0; q < kSeg; ++q) v += cnt[q * M + j];
  ptr[j] = v;
}

__global__ void __launch_bounds__(1024) k_cg_csc_scan(int64_t M, int64_t* ptr) {
  // in place: each thread reads each of its entries before writing it
  __shared__ int64_t part[1024];
  const int t = threadIdx.x;
  const int64_t per = (M + 1023) / 1024;
  const int64_t i0 = t * per, i1 = i0 + per < M ? i0 + per : M;
  int64_t s = 0;
  for (int64_t i = i0; i < i1; ++i) s += ptr[i];
  part[t] = s;
  __syncthreads();
  if (t == 0) {
    int64_t run = 0;
    for (int i = 0; i < 1024; ++i) {
      const int64_t x = part[i];
      part[i] = run;
      run += x;
    }
    ptr[M] = run;
  }
  __syncthreads();
  int64_t run = part[t];
  for (int64_t i = i0; i < i1; ++i) {
    const int64_t x = ptr[i];
    ptr[i] = run;
    run += x;
  }
}

__global__ void __launch_bounds__(256) k_cg_csc_fill(const uint64_t* __restrict__ T, int64_t M, int64_t nrb_s,
                                                     const int64_t* __restrict__ ptr, const int32_t* __restrict__ cnt,
                                                     int64_t nnz, int32_t* __restrict__ rows) {
  const int64_t j = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const int sg = blockIdx.y;
  if (j >= M) return;
  int64_t pos = ptr[j];
  for (int q = 0; q < sg; ++q) pos += cnt[q * M + j];
  const int64_t end = ptr[j + 1] < nnz ? ptr[j + 1] : nnz;
  const int64_t r0 = nrb_s * sg / kSeg, r1 = nrb_s * (sg + 1) / kSeg;
  for (int64_t rb = r0; rb < r1; ++rb) {
    uint64_t word = T[rb * M + j];
    while (word && pos < end) {
      rows[pos++] = static_cast<int32_t>(rb * 64 + __builtin_ctzll(word));
      word &= word - 1;
    }
  }
}

// Update of iteration t (see the recurrences above); partial gamma_{t+1}.
__global__ void __launch_bounds__(256) k_cg_update(GroupArgs g) {
  __shared__ double red[4];
  __shared__ double coef[3];
  int64_t bid;
  const int m = member_of(g, bid);
  const Args& a = g.a[m];
  const int64_t t = g.t[m];
  if (a.st->done) return;
  const int64_t j = bid * 256 + threadIdx.x;
  // this thread's vector entries first: their loads overlap the scalar sums
  double q = 0.0, rj = 0.0, pj = 0.0, sj = 0.0;
  if (j < a.M) {
    if (a.has_random) {
      if (a.rs > 0) q = a.qs[j];
      q = chunk_sum(a.qpart + j, a.M, a.nrcd, q);
    }
    rj = a.r[j];
    pj = a.p[j];
    sj = a.s[j];
  }
  // the four scalar sums, one per wavefront, side by side
  __shared__ double sums[4];
  {
    const int wv = threadIdx.x >> 6;
    double v = 0.0;
    if (wv == 0) v = wave_fixed_sum(a.rr + (t % 3) * a.nbc, a.nbc);
    else if (wv == 1) v = a.has_random ? wave_fixed_sum(a.uu, a.nbu, 2) : 0.0;
    else if (wv == 2) v = a.has_random ? wave_fixed_sum(a.uu + 1, a.nbu, 2) : 0.0;
    else v = t > 0 ? wave_fixed_sum(a.rr + ((t + 2) % 3) * a.nbc, a.nbc) : 1.0;
    if ((threadIdx.x & 63) == 0) sums[wv] = v;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    const double g = sums[0], uu = sums[1], su = sums[2], gp = sums[3];
    const double delta = a.alpha * g + a.wr2 * uu;
    double beta = 0.0, den = delta;
    if (t > 0) {
      beta = g / gp;
      den = delta - beta * g / a.hist[(t + 1) & 1];
    }
    const double step = g / den;
    const bool ok = den > 0.0 && step == step && step < 1e300 && beta == beta;
    coef[0] = ok ? step : -1.0;
    coef[1] = beta;
    coef[2] = su / static_cast<double>(a.M);
    if (ok && bid == 0) a.hist[t & 1] = step;
  }
  __syncthreads();
  const double step = coef[0], beta = coef[1], mq = coef[2];
  if (step < 0.0) {   // identical in every workgroup
    if (bid == 0 && threadIdx.x == 0) {
      a.st->done = 1;
      a.st->iters = static_cast<int32_t>(t);
      a.st->status = 2;
      __hip_atomic_store(a.host_flag + 1, static_cast<int32_t>(t), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
      __hip_atomic_store(a.host_flag, 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
    }
    return;
  }
  double r2 = 0.0;
  if (j < a.M) {
    const double wj = a.alpha * rj + a.wr2 * (q - mq);
    const double pn = rj + beta * pj;
    const double sn = wj + beta * sj;
    a.p[j] = pn;
    a.s[j] = sn;
    a.x[j] += step * pn;
    const double rn = rj - step * sn;
    a.r[j] = rn;
    r2 = rn * rn;
  }
  const double sb = block_sum_d(r2, red);
  if (threadIdx.x == 0) a.rr[((t + 1) % 3) * a.nbc + bid] = sb;
}

// phi = Delta/M + x - mean(x) (the projection made exact), info from the state.
__global__ void __launch_bounds__(1024) k_cg_finish(const double* __restrict__ x, int64_t M,
                                                    const gnnshap::CgState* __restrict__ st,
                                                    const float* __restrict__ fef, float* __restrict__ phi,
                                                    int32_t* info, int32_t undetermined) {
  __shared__ double red[16];
  double sm = 0.0;
  for (int64_t j = threadIdx.x; j < M; j += 1024) sm += x[j];
  const double mean = block_sum_d(sm, red) / static_cast<double>(M);
  const double base = (static_cast<double>(fef[1]) - static_cast<double>(fef[0])) / static_cast<double>(M);
  for (int64_t j = threadIdx.x; j < M; j += 1024) phi[j] = static_cast<float>(base + (x[j] - mean));
  if (threadIdx.x == 0) *info = (st->status == 0 && !undetermined) ? 0 : static_cast<int32_t>(M + 1);
}

// Mapped page-locked stopping flags of the calling thread and their device
// addresses: one slot per solve in flight (created on first use, kept until
// the process ends).
struct HostFlag {
  int32_t* host = nullptr;
  int32_t* dev = nullptr;
  bool busy = false;
};

constexpr int kFlagSlots = 16;

HostFlag* acquire_flag() {
  static thread_local HostFlag pool[kFlagSlots];
  for (HostFlag& f : pool) {
    if (f.busy) continue;
    if (!f.host) {
      void* h = nullptr;
      if (hipHostMalloc(&h, 256, hipHostMallocMapped | hipHostMallocCoherent) != hipSuccess) {
        (void)hipGetLastError();
        return nullptr;
      }
      void* d = nullptr;
      if (hipHostGetDevicePointer(&d, h, 0) != hipSuccess) {
        (void)hipGetLastError();
        (void)hipHostFree(h);
        return nullptr;
      }
      f.host = static_cast<int32_t*>(h);
      f.dev = static_cast<int32_t*>(d);
    }
    f.busy = true;
    return &f;
  }
  return nullptr;
}

// The two events of a group's chunk ring, per calling thread (created on
// first use, kept until the process ends).
struct EventPair {
  hipEvent_t ev[2] = {nullptr, nullptr};
  bool busy = false;
};

constexpr int kPairSlots = 8;

EventPair* acquire_pair() {
  static thread_local EventPair pool[kPairSlots];
  for (EventPair& e : pool) {
    if (e.busy) continue;
    for (int i = 0; i < 2; ++i)
      if (!e.ev[i] && hipEventCreateWithFlags(&e.ev[i], hipEventDisableTiming) != hipSuccess) {
        (void)hipGetLastError();
        return nullptr;
      }
    e.busy = true;
    return &e;
  }
  return nullptr;
}

// Whether the work recorded by ev has completed, without waiting; a query
// that finds it pending leaves no error behind for the next launch check.
bool event_done(hipEvent_t ev) {
  const hipError_t e = hipEventQuery(ev);
  if (e == hipErrorNotReady) {
    (void)hipGetLastError();
    return false;
  }
  return true;   // complete, or an error that the wait on it reports
}

}  // namespace

gnnshap::CgShape gnnshap::cg_shape(int64_t M, int64_t wpr, int64_t kr, int64_t rb0, const gnnshap_class* classes,
                                   int64_t ncls) {
  CgShape s{};
  s.M = M;
  s.wpr = wpr;
  s.kr = kr;
  s.nrb = ceil_div(kr, 64);
  // sparse rows: the longest run of random rows from the first whose sizes are
  // at most M / kSparseDiv, cut to whole 64-row groups
  if (kr > 0 && classes) {
    const int64_t tmax = M / kSparseDiv;
    std::vector<int32_t> sz;
    sz.reserve(static_cast<size_t>(kr));
    for (int64_t i = 0; i < ncls && static_cast<int64_t>(sz.size()) < kr; ++i) {
      if (classes[i].row_begin + classes[i].row_count <= rb0) continue;
      if (classes[i].size > tmax) break;
      const int64_t from = std::max<int64_t>(classes[i].row_begin, rb0);
      for (int64_t r = from; r < classes[i].row_begin + classes[i].row_count; ++r) sz.push_back(classes[i].size);
    }
    s.rs = (std::min<int64_t>(static_cast<int64_t>(sz.size()), kr) / 64) * 64;
    if (s.rs > 64 * 1024) s.rs = 64 * 1024;   // the item table's scan holds 1024 blocks
    for (int64_t b = 0; b < s.rs; ++b) s.nnz += sz[b];
    for (int64_t q = 0; q < s.rs / 64; ++q) s.nsi += int64_t(1) << sparse_lanes_log2(sz[64 * q + 63]);
  }
  s.rbd0 = s.rs / 64;
  const int64_t nrbd = std::max<int64_t>(s.nrb - s.rbd0, 1);
  // pass A: at least kFill (row block, player chunk) pairs, chunks of whole
  // words, at most kTabA words of tables per workgroup
  const int64_t npc = std::max<int64_t>(ceil_div(wpr, kTabA), std::min(ceil_div(kFill, nrbd), wpr));
  s.pwords = ceil_div(wpr, npc);
  s.npc = ceil_div(wpr, s.pwords);
  // pass B: at least kFill (player word, row chunk) pairs, chunks of whole
  // row blocks, at most kTabB row blocks of tables per workgroup
  const int64_t nrc = std::max<int64_t>(ceil_div(nrbd, kTabB), std::min(ceil_div(kFill, wpr), nrbd));
  s.rbc = ceil_div(nrbd, nrc);
  s.nrc = ceil_div(nrbd, s.rbc);
  // workgroups of the sparse rows in pass A (rows) and pass B (players), at
  // most 2048 each (each wave loops), and of the bit rows in the row pass
  s.nsa = s.rs > 0 ? std::min<int64_t>(ceil_div(s.nsi, kWaves), 2048) : 0;
  // pass B: lanes per player list from the mean list length (longer lists loop)
  s.lgb = sparse_lanes_log2(ceil_div(s.nnz, M));
  s.nsb = s.rs > 0 ? std::min<int64_t>(ceil_div(ceil_div(M, int64_t(64) >> s.lgb), kWaves), 2048) : 0;
  s.nrcd = s.rbd0 < s.nrb ? s.nrc : 0;
  s.nbu = 1 + ceil_div(kr - s.rs > 0 ? kr - s.rs : 1, 256);
  s.nbc = ceil_div(wpr * 64, 256);
  return s;
}

gnnshap::CgWs gnnshap::cg_carve(Carver& c, const CgShape& sh) {
  CgWs w;
  const int64_t kr = sh.kr > 0 ? sh.kr : 1;
  w.x = c.take<double>(sh.M);
  w.r = c.take<double>(sh.wpr * 64);
  w.p = c.take<double>(sh.M);
  w.s = c.take<double>(sh.M);
  w.upart = c.take<double>(sh.npc * kr);
  w.u = c.take<double>((sh.nrb > 0 ? sh.nrb : 1) * 64);
  w.qpart = c.take<double>(sh.nrc * sh.M);
  w.uu = c.take<double>(2 * sh.nbu);
  w.usp = c.take<double>(2 * (sh.nsa > 0 ? sh.nsa : 1));
  w.rr = c.take<double>(3 * sh.nbc);
  w.hist = c.take<double>(2);
  w.sz = c.take<int32_t>(kr);
  w.blocked = c.take<uint64_t>((sh.nrb > 0 ? sh.nrb : 1) * sh.wpr * 64);
  w.st = c.take<CgState>(1);
  w.csr_ptr = c.take<int64_t>(sh.rs + 1);
  w.csr_idx = c.take<int32_t>(sh.nnz > 0 ? sh.nnz : 1);
  w.csc_ptr = c.take<int64_t>(sh.M + 1);
  w.csc_row = c.take<int32_t>(sh.nnz > 0 ? sh.nnz : 1);
  w.qs = c.take<double>(sh.M);
  w.sitem = c.take<int64_t>(sh.nsi > 0 ? sh.nsi : 1);
  w.segcnt = c.take<int32_t>(kSeg * std::max<int64_t>(std::max<int64_t>(sh.rs, sh.M), 1));
  return w;
}

// One member of a group: its arguments, shape, problem and flag, the
// iteration its next launch runs and its grids.
struct Member {
  Args a;
  gnnshap::CgShape sh;
  gnnshap::CgProblem pr;
  gnnshap::CgWs w;
  HostFlag* hf = nullptr;
  int64_t t = 0;
  uint32_t ga = 0, gb = 0, g_rows = 0, g_upd = 0;
};

// pw row blocks (pass A) and player words (pass B) per wavefront: the
// passes' grids follow; the sums, and so the results, do not depend on pw.
void set_per_wave(Member& m, int pw) {
  Args& a = m.a;
  const gnnshap::CgShape& sh = m.sh;
  a.pw = pw;
  a.nxa = gnnshap::ceil_div(std::max<int64_t>(sh.nrb - sh.rbd0, 1), kWaves * pw);
  a.nxb = gnnshap::ceil_div(sh.wpr, kWaves * pw);
  m.ga = static_cast<uint32_t>(a.nxa * sh.npc + sh.nsa);
  m.gb = static_cast<uint32_t>(a.nxb * sh.nrcd + sh.nsb);
}

struct gnnshap::CgGroup::State {
  std::vector<Member> mem;
  EventPair* ev = nullptr;
  int64_t chunk = 0;
};

gnnshap::CgGroup::CgGroup() : st_(new State()) {}

gnnshap::CgGroup::~CgGroup() {
  for (Member& m : st_->mem)
    if (m.hf) m.hf->busy = false;
  if (st_->ev) st_->ev->busy = false;
}

int gnnshap::CgGroup::size() const { return static_cast<int>(st_->mem.size()); }

int gnnshap::CgGroup::add(const CgProblem& pr, const CgShape& sh, const CgWs& w) {
  State& S = *st_;
  if (full()) return fail(GNNSHAP_EINVAL, "solver group already holds %d systems", kCgGroupMax);
  if (!S.ev) {
    S.ev = acquire_pair();
    if (!S.ev) return fail(GNNSHAP_EHIP, "could not create the solver's events (or more than %d groups)", kPairSlots);
  }
  HostFlag* hf = acquire_flag();
  if (!hf) return fail(GNNSHAP_EHIP, "could not allocate the solver's host flag (or more than %d solves in flight)",
                       kFlagSlots);
  hipStream_t s = s_;
  Member m;
  m.hf = hf;
  m.sh = sh;
  m.pr = pr;
  m.w = w;
  Args& a = m.a;
  a = Args{};
  a.blocked = pr.blocked;
  a.T = pr.T;
  a.sz = w.sz;
  a.M = sh.M;
  a.wpr = sh.wpr;
  a.kr = sh.kr;
  a.nrb = sh.nrb;
  a.npc = sh.npc;
  a.pwords = sh.pwords;
  a.nrc = sh.nrc;
  a.rbc = sh.rbc;
  a.nbu = sh.nbu;
  a.nbc = sh.nbc;
  a.alpha = pr.alpha;
  a.wr2 = sh.kr > 0 ? 2.0 * pr.wr : 0.0;
  a.tol2 = kTol * kTol;
  a.maxit = kMaxIt;
  a.has_random = sh.kr > 0 ? 1 : 0;
  a.x = w.x;
  a.r = w.r;
  a.p = w.p;
  a.s = w.s;
  a.upart = w.upart;
  a.u = w.u;
  a.qpart = w.qpart;
  a.uu = w.uu;
  a.usp = w.usp;
  a.rr = w.rr;
  a.hist = w.hist;
  a.st = w.st;
  a.rs = sh.rs;
  a.rbd0 = sh.rbd0;
  a.nsa = sh.nsa;
  a.nsi = sh.nsi;
  a.lgb = sh.lgb;
  a.sitem = w.sitem;
  a.nsb = sh.nsb;
  a.nrcd = sh.nrcd;
  set_per_wave(m, 1);
  a.csr_ptr = w.csr_ptr;
  a.csr_idx = w.csr_idx;
  a.csc_ptr = w.csc_ptr;
  a.csc_row = w.csc_row;
  a.qs = w.qs;
  a.host_flag = hf->dev;
  m.g_rows = static_cast<uint32_t>(sh.nbu);
  m.g_upd = static_cast<uint32_t>(sh.nbc);
  // no kernel of an earlier solve that used this flag writes it any more:
  // a solve stops writing it at its stopping iteration, which had completed
  // before the flag was released
  __atomic_store_n(hf->host, 0, __ATOMIC_RELEASE);
  __atomic_store_n(hf->host + 1, -1, __ATOMIC_RELEASE);
  {
    GS_TIMED("k_cg_init", s);
    k_cg_init<<<static_cast<unsigned>(sh.nbc), 256, 0, s>>>(a, pr.dv, pr.bsum, pr.nb, pr.classes, pr.ncls, pr.rb0,
                                                            w.sz);
  }
  GS_LAUNCHED();
  if (sh.rs > 0) {
    // the sparse rows' lists (row sizes from k_cg_init); qs serves as the
    // count scratch here, it is written before the iterations read it
    const int64_t nrb_s = sh.rs / 64;
    const dim3 gr(static_cast<unsigned>(nrb_s), kSeg), gp(static_cast<unsigned>(ceil_div(sh.M, 256)), kSeg);
    GS_TIMED("k_cg_sparse_build", s);
    k_cg_csr_ptr<<<1, 1024, 0, s>>>(w.sz, sh.rs, w.csr_ptr, w.sitem);
    GS_LAUNCHED();
    k_cg_csr_count<<<gr, 64, 0, s>>>(pr.blocked, sh.wpr, sh.rs, w.segcnt);
    GS_LAUNCHED();
    k_cg_csr_fill<<<gr, 64, 0, s>>>(pr.blocked, sh.wpr, sh.rs, w.csr_ptr, w.segcnt, sh.nnz, w.csr_idx);
    GS_LAUNCHED();
    k_cg_csc_count<<<gp, 256, 0, s>>>(pr.T, sh.M, nrb_s, w.segcnt);
    GS_LAUNCHED();
    k_cg_csc_total<<<static_cast<unsigned>(ceil_div(sh.M, 256)), 256, 0, s>>>(w.segcnt, sh.M, w.csc_ptr);
    GS_LAUNCHED();
    k_cg_csc_scan<<<1, 1024, 0, s>>>(sh.M, w.csc_ptr);
    GS_LAUNCHED();
    k_cg_csc_fill<<<gp, 256, 0, s>>>(pr.T, sh.M, nrb_s, w.csc_ptr, w.segcnt, sh.nnz, w.csc_row);
    GS_LAUNCHED();
  }
  S.mem.push_back(m);
  return GNNSHAP_OK;
}

bool gnnshap::CgGroup::ready() const {
  const State& S = *st_;
  return S.chunk < 2 || event_done(S.ev->ev[S.chunk & 1]);   // step() waits for the chunk before last
}

namespace {

// Fills g with the members selected by `take` (grid of member m: grid(m)),
// each at iteration t + dt; returns the total number of workgroups.
template <class Take, class Grid>
uint32_t fill_group(GroupArgs& g, const std::vector<Member>& mem, int64_t dt, Take take, Grid grid) {
  g.n = 0;
  uint32_t total = 0;
  for (const Member& m : mem) {
    if (!take(m, m.t + dt)) continue;
    g.a[g.n] = m.a;
    g.t[g.n] = m.t + dt;
    g.blk[g.n] = total;
    total += grid(m);
    ++g.n;
  }
  g.blk[g.n] = total;
  return total;
}

}  // namespace

// Waits for the chunk before the last one queued; every member whose stop
// flag is set gets phi and info queued (after the chunks already queued,
// whose launches it leaves at once) and leaves the group.  Then queues
// iterations t .. t + kChunk - 1 of every member left (pass A alone of
// iteration kMaxIt, which always stops; nothing beyond it) and records the
// chunk's event.  The ring has two events: chunk n reuses the event of chunk
// n - 2, which has completed by then.
int gnnshap::CgGroup::step() {
  State& S = *st_;
  if (S.mem.empty()) return GNNSHAP_OK;
  hipStream_t s = s_;
  if (S.chunk >= 2) {
    GS_HIP(hipEventSynchronize(S.ev->ev[S.chunk & 1]));
    for (size_t i = 0; i < S.mem.size();) {
      Member& m = S.mem[i];
      if (__atomic_load_n(m.hf->host, __ATOMIC_ACQUIRE) == 0) {
        ++i;
        continue;
      }
      const int64_t iters = __atomic_load_n(m.hf->host + 1, __ATOMIC_ACQUIRE);
      last_iters_ = iters;
      const CgShape& sh = m.sh;
      timing_note_solve(sh.M, sh.wpr, sh.kr, iters, sh.rs, sh.nnz);
      {
        GS_TIMED("k_cg_finish", s);
        // without enumerated classes, fewer than M - 1 random rows cannot
        // determine psi (1-perp has M - 1 dimensions): reported like a failed pivot
        const int32_t undetermined = (m.pr.alpha == 0.0 && sh.kr < sh.M - 1) ? 1 : 0;
        k_cg_finish<<<1, 1024, 0, s>>>(m.w.x, sh.M, m.w.st, m.pr.fef, m.pr.phi, m.pr.info, undetermined);
      }
      GS_LAUNCHED();
      m.hf->busy = false;
      S.mem.erase(S.mem.begin() + static_cast<std::ptrdiff_t>(i));
    }
    if (S.mem.empty()) return GNNSHAP_OK;
  }
  // a system alone fills the GPU better with one row block (player word)
  // per wavefront, several systems leave fewer, longer wavefronts
  const int pw = S.mem.size() >= 2 ? kPerWaveGroup : 1;
  for (Member& m : S.mem)
    if (m.a.pw != pw) set_per_wave(m, pw);
  GroupArgs g;
  for (int64_t dt = 0; dt < kChunk; ++dt) {
    uint32_t n = fill_group(g, S.mem, dt, [](const Member&, int64_t t) { return t <= kMaxIt; },
                            [](const Member& m) { return m.ga; });
    if (g.n == 0) break;
    {
      GS_TIMED("k_cg_pass_a", s);
      if (pw == 1)
        k_cg_pass_a<1><<<n, kWaves * 64, 0, s>>>(g);
      else
        k_cg_pass_a<kPerWaveGroup><<<n, kWaves * 64, 0, s>>>(g);
    }
    GS_LAUNCHED();
    n = fill_group(g, S.mem, dt, [](const Member& m, int64_t t) { return t < kMaxIt && m.sh.kr > 0; },
                   [](const Member& m) { return m.g_rows; });
    if (g.n > 0) {
      {
        GS_TIMED("k_cg_rows", s);
        k_cg_rows<<<n, 256, 0, s>>>(g);
      }
      GS_LAUNCHED();
      n = fill_group(g, S.mem, dt, [](const Member& m, int64_t t) { return t < kMaxIt && m.sh.kr > 0; },
                     [](const Member& m) { return m.gb; });
      {
        GS_TIMED("k_cg_pass_b", s);
        if (pw == 1)
          k_cg_pass_b<1><<<n, kWaves * 64, 0, s>>>(g);
        else
          k_cg_pass_b<kPerWaveGroup><<<n, kWaves * 64, 0, s>>>(g);
      }
      GS_LAUNCHED();
    }
    n = fill_group(g, S.mem, dt, [](const Member&, int64_t t) { return t < kMaxIt; },
                   [](const Member& m) { return m.g_upd; });
    if (g.n > 0) {
      {
        GS_TIMED("k_cg_update", s);
        k_cg_update<<<n, 256, 0, s>>>(g);
      }
      GS_LAUNCHED();
    }
  }
  for (Member& m : S.mem) m.t = std::min(m.t + kChunk, kMaxIt + 1);
  GS_HIP(hipEventRecord(S.ev->ev[S.chunk & 1], s));
  ++S.chunk;
  return GNNSHAP_OK;
}

int gnnshap::cg_solve(const CgProblem& pr, const CgShape& sh, const CgWs& w, hipStream_t s, int64_t* iters_out) {
  CgGroup grp;
  grp.set_stream(s);
  if (int st = grp.add(pr, sh, w)) return st;
  while (!grp.empty())
    if (int st = grp.step()) return st;
  if (iters_out) *iters_out = grp.last_iters();
  return GNNSHAP_OK;
}
