// Constrained Kernel-SHAP weighted least squares (eq. 2-3, Alg. 1 step 5 and
// Sec. 3.5 of the GNNShap paper).
//
// Minimise sum_b w_b (y_b - f0 - m_b.phi)^2 subject to sum(phi) = Delta =
// f(E_c) - f0.  With phi = Delta/M 1 + psi, 1.psi = 0 and P = I - 11^T/M the
// normal equations become  (P G P + gamma 11^T/M) psi = P (r - Delta/M G 1),
// G = sum_b w_b m_b m_b^T, r = sum_b w_b (y_b - f0) m_b; the shift gamma =
// tr(PGP)/(M-1) makes the system positive definite without changing psi.
//
// The plan's structure makes G exact and cheap:
//   * a row and its complement give P(m m^T + mbar mbar^T)P = 2 P m m^T P;
//   * an enumerated class of size c contributes w_c kappa_c C(M-2, c-1) P
//     (all c-subsets: diagonal C(M-1,c-1), off-diagonal C(M-2,c-2));
//   * the random rows share one weight w_r, so their part is 2 w_r P C_R P
//     with C_R the integer co-occurrence counts of the random representative
//     rows, computed exactly by popcounts on a bit-transposed copy.
// Systems whose lower triangle fits in LDS are assembled, factored and solved
// by one workgroup; larger ones use a blocked right-looking Cholesky over the
// whole GPU (64-wide panels) and one workgroup for the two triangular solves.
// Diagonal blocks are factored by one wavefront holding a row per lane in
// registers; tail blocks are padded with the identity so every inner loop
// runs without per-lane branches.  The right-hand side is accumulated in fp64.
#include <cmath>

#include "common.h"

namespace {

constexpr int kNB = 64;   // panel width, multi-block path
constexpr int kSB = 32;   // panel width, one-workgroup path
constexpr int kMaxChunks = 256;

struct Ws {
  gnnshap_class* classes;
  uint64_t* T;       // nrb x M: bit b of T[rb, j] = player j in random row rb*64+b
  float* G;          // M x M (int32 counts first, then the system, lower part factored)
  int64_t* usum;     // M: row sums of the counts
  double* scal;      // [0] trace, [1] sigma, [2] gamma, [3] delta, [4] f0
  double* part;      // nch x M partial right-hand sides
  float* rhs;        // M
  float* x;          // M
  float* Ld;         // kNB x kNB padded diagonal factor + kNB reciprocal pivots
};

int64_t n_chunks(int64_t half) {
  int64_t c = gnnshap::ceil_div(half, 256);
  return c < 1 ? 1 : (c > kMaxChunks ? kMaxChunks : c);
}

Ws carve(gnnshap::Carver& c, const gnnshap_sample_plan* p) {
  Ws w;
  const int64_t M = p->num_players;
  const int64_t half = p->num_rows / 2;
  const int64_t kr = half - p->random_begin;
  const int64_t nrb = gnnshap::ceil_div(kr, 64);
  w.classes = c.take<gnnshap_class>(p->num_classes > 0 ? p->num_classes : 1);
  w.T = c.take<uint64_t>((nrb > 0 ? nrb : 1) * M);
  w.G = c.take<float>(M * M);
  w.usum = c.take<int64_t>(M);
  w.scal = c.take<double>(16);
  w.part = c.take<double>(n_chunks(half) * M);
  w.rhs = c.take<float>(M);
  w.x = c.take<float>(M);
  w.Ld = c.take<float>(kNB * kNB + kNB);
  return w;
}

__device__ inline float bcast(float v, int lane) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}

// a[lane] without a dynamic register index: unrolled selects.
template <int NB>
__device__ inline float lane_entry(const float (&a)[NB]) {
  const int lane = threadIdx.x & 63;
  float d = 1.f;
#pragma unroll
  for (int c = 0; c < NB; ++c) d = c == lane ? a[c] : d;
  return d;
}

// Cholesky of an NB x NB lower block held by one wavefront, row `lane` in
// a[] (rows and columns past the real block are the identity).  Column k:
// broadcast the pivot, scale the column, rank-1 update of the later
// columns.  Entries above each lane's diagonal are left undefined.  The
// first non-positive pivot (1-based, offset o) goes to *info and is replaced
// by 1.
template <int NB>
__device__ inline void chol_regs(float (&a)[NB], int64_t o, int32_t* info) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int k = 0; k < NB; ++k) {
    float piv = bcast(a[k], k);
    if (!(piv > 0.f)) {
      if (lane == 0) atomicCAS(info, 0, static_cast<int32_t>(o + k + 1));
      piv = 1.f;
    }
    // lane k holds the pivot itself: piv / sqrt(piv) = sqrt(piv), so one
    // scaling serves the diagonal and the column below it
    a[k] *= 1.0f / sqrtf(piv);
#pragma unroll
    for (int j = k + 1; j < NB; ++j) a[j] -= a[k] * bcast(a[k], j);
  }
}

// T[rb, j]: transpose 64 rows x 64 players with ballots.  One wave per (rb, word).
__global__ void __launch_bounds__(64) k_transpose(const uint64_t* __restrict__ masks, int64_t wpr,
                                                  int64_t row0, int64_t nrows, int64_t M,
                                                  uint64_t* __restrict__ T) {
  const int lane = threadIdx.x;
  const int64_t rb = blockIdx.x;
  const int64_t w = blockIdx.y;
  const int64_t r = rb * 64 + lane;
  const uint64_t word = r < nrows ? masks[(row0 + r) * wpr + w] : 0;
  uint64_t mine = 0;
#pragma unroll 8
  for (int p = 0; p < 64; ++p) {
    const uint64_t bal = __ballot((word >> p) & 1);
    if (lane == p) mine = bal;
  }
  const int64_t j = w * 64 + lane;
  if (j < M) T[rb * M + j] = mine;
}

// Counts C[i, j] = sum_rb popcount(T[rb, i] & T[rb, j]) for 64x64 tiles with J >= I,
// stored in both halves.
__global__ void __launch_bounds__(256) k_gram(const uint64_t* __restrict__ T, int64_t nrb, int64_t M,
                                              int32_t* __restrict__ C) {
  const int64_t I = blockIdx.y, J = blockIdx.x;
  if (J < I) return;
  __shared__ uint64_t Ti[16][64];
  __shared__ uint64_t Tj[16][64];
  const int tid = threadIdx.x;
  const int ty = tid / 16, tx = tid % 16;
  int acc[4][4] = {};
  for (int64_t k0 = 0; k0 < nrb; k0 += 16) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int idx = tid + q * 256;
      const int kk = idx / 64, c = idx % 64;
      const int64_t i = I * 64 + c, j = J * 64 + c;
      const bool kin = k0 + kk < nrb;
      Ti[kk][c] = (kin && i < M) ? T[(k0 + kk) * M + i] : 0;
      Tj[kk][c] = (kin && j < M) ? T[(k0 + kk) * M + j] : 0;
    }
    __syncthreads();
#pragma unroll 4
    for (int kk = 0; kk < 16; ++kk) {
      uint64_t a[4], b[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        a[q] = Ti[kk][ty * 4 + q];
        b[q] = Tj[kk][tx * 4 + q];
      }
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[q][r] += __popcll(a[q] & b[r]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int64_t i = I * 64 + ty * 4 + q;
    if (i >= M) continue;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t j = J * 64 + tx * 4 + r;
      if (j >= M) continue;
      C[i * M + j] = acc[q][r];
      C[j * M + i] = acc[q][r];
    }
  }
}

// usum[i] = sum_j C[i, j]; one wave per row.
__global__ void __launch_bounds__(256) k_rowsum(const int32_t* __restrict__ C, int64_t M,
                                                int64_t* __restrict__ usum) {
  const int lane = threadIdx.x & 63;
  const int64_t i = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) >> 6;
  if (i >= M) return;
  long long s = 0;
  for (int64_t j = lane; j < M; j += 64) s += C[i * M + j];
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
  if (lane == 0) usum[i] = s;
}

// scal: trace and sigma of the counts (exact), gamma, Delta, f0.  One block.
__global__ void __launch_bounds__(256) k_scalars(const int32_t* __restrict__ C, const int64_t* __restrict__ usum,
                                                 int64_t M, bool has_random, double alpha, double wr,
                                                 const float* __restrict__ fef, double* scal) {
  __shared__ long long st[256], ss[256];
  const int tid = threadIdx.x;
  long long tr = 0, sg = 0;
  if (has_random)
    for (int64_t i = tid; i < M; i += 256) {
      tr += C[i * M + i];
      sg += usum[i];
    }
  st[tid] = tr;
  ss[tid] = sg;
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if (tid < off) {
      st[tid] += st[tid + off];
      ss[tid] += ss[tid + off];
    }
    __syncthreads();
  }
  if (tid == 0) {
    const double Md = static_cast<double>(M);
    const double trace = static_cast<double>(st[0]);
    const double sigma = static_cast<double>(ss[0]);
    const double tr_pgp = alpha * (Md - 1.0) + 2.0 * wr * (trace - sigma / Md);
    scal[0] = trace;
    scal[1] = sigma;
    scal[2] = tr_pgp / (Md - 1.0);
    scal[3] = static_cast<double>(fef[1]) - static_cast<double>(fef[0]);
    scal[4] = static_cast<double>(fef[0]);
  }
}

// In place: counts (int32) -> G~ (fp32), lower and upper.
__global__ void __launch_bounds__(256) k_build(float* G, const int64_t* __restrict__ usum, int64_t M,
                                               bool has_random, double alpha, double wr,
                                               const double* __restrict__ scal) {
  const double Md = static_cast<double>(M);
  const double sigma = scal[1], gamma = scal[2];
  const int64_t total = M * M;
  for (int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; t < total;
       t += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const int64_t i = t / M, j = t % M;
    double v = alpha * ((i == j ? 1.0 : 0.0) - 1.0 / Md) + gamma / Md;
    if (has_random) {
      const double cij = static_cast<double>(reinterpret_cast<const int32_t*>(G)[t]);
      v += 2.0 * wr * (cij - static_cast<double>(usum[i] + usum[j]) / Md + sigma / (Md * Md));
    }
    G[t] = static_cast<float>(v);
  }
}

// Partial right-hand sides: part[ch, j] = sum_{b in chunk ch} dz_b m_bj with
// dz_b = z_b - z_{b+half}, z_b = w_b (y_b - f0 - Delta/M |S_b|), b < half.
__global__ void __launch_bounds__(256) k_rhs_part(const uint64_t* __restrict__ masks, int64_t wpr,
                                                  int64_t half, int64_t M, const float* __restrict__ y,
                                                  const gnnshap_class* __restrict__ cls, int64_t ncls,
                                                  const float* __restrict__ fef, int64_t rows_per_chunk,
                                                  double* __restrict__ part) {
  __shared__ double dzs[256];
  const int tid = threadIdx.x;
  const int64_t r0 = static_cast<int64_t>(blockIdx.x) * rows_per_chunk;
  const int64_t r1 = r0 + rows_per_chunk < half ? r0 + rows_per_chunk : half;
  const double Md = static_cast<double>(M);
  const double f0 = static_cast<double>(fef[0]);
  const double delta = static_cast<double>(fef[1]) - f0;
  for (int64_t j0 = 0; j0 < M; j0 += 256) {
    const int64_t j = j0 + tid;
    double acc = 0.0;
    for (int64_t b0 = r0; b0 < r1; b0 += 256) {
      const int nb = static_cast<int>(r1 - b0 < 256 ? r1 - b0 : 256);
      __syncthreads();
      if (tid < nb) {
        const int64_t b = b0 + tid;
        int64_t lo = 0, hi = ncls - 1;
        while (lo < hi) {
          const int64_t mid = (lo + hi + 1) >> 1;
          if (cls[mid].row_begin <= b) lo = mid; else hi = mid - 1;
        }
        const double w = cls[lo].weight;
        const int64_t pc = cls[lo].size;               // |S_b|: representatives have their class size
        const double z1 = w * (static_cast<double>(y[b]) - f0 - delta / Md * static_cast<double>(pc));
        const double z2 = w * (static_cast<double>(y[b + half]) - f0 - delta / Md * static_cast<double>(M - pc));
        dzs[tid] = z1 - z2;
      }
      __syncthreads();
      if (j < M) {
        const uint64_t* col = masks + b0 * wpr + (j >> 6);
        const int sh = static_cast<int>(j & 63);
        for (int q = 0; q < nb; ++q)
          if ((col[q * wpr] >> sh) & 1) acc += dzs[q];
      }
    }
    if (j < M) part[static_cast<int64_t>(blockIdx.x) * M + j] = acc;
  }
}

// rhs = P (sum of the partials); one block.
__global__ void __launch_bounds__(1024) k_rhs_finish(const double* __restrict__ part, int64_t nch, int64_t M,
                                                     float* __restrict__ rhs, double* scal) {
  __shared__ double red[1024];
  const int tid = threadIdx.x;
  double s = 0.0;
  for (int64_t j = tid; j < M; j += 1024) {
    double v = 0.0;
    for (int64_t c = 0; c < nch; ++c) v += part[c * M + j];
    s += v;
  }
  red[tid] = s;
  __syncthreads();
  for (int off = 512; off > 0; off >>= 1) {
    if (tid < off) red[tid] += red[tid + off];
    __syncthreads();
  }
  const double mean = red[0] / static_cast<double>(M);
  for (int64_t j = tid; j < M; j += 1024) {
    double v = 0.0;
    for (int64_t c = 0; c < nch; ++c) v += part[c * M + j];
    rhs[j] = static_cast<float>(v - mean);
  }
}

// One-workgroup path: the lower triangle of G~ packed in LDS (row i at
// i(i+1)/2).
__device__ inline int64_t tri(int64_t i, int64_t j) { return ((i * (i + 1)) >> 1) + j; }

size_t small_lds_bytes(int64_t M) {
  return static_cast<size_t>(M) * (sizeof(double) + 2 * sizeof(float)) +
         static_cast<size_t>((M * (M + 1)) / 2) * sizeof(float);
}

__global__ void __launch_bounds__(256) k_solve_small(const int32_t* __restrict__ C, int64_t M, bool has_random,
                                                     double alpha, double wr, const float* __restrict__ fef,
                                                     const double* __restrict__ part, int64_t nch,
                                                     int32_t* info, float* __restrict__ phi) {
  extern __shared__ __align__(16) unsigned char smem[];
  double* dv = reinterpret_cast<double*>(smem);      // M: row sums, then the raw right-hand side
  float* rhs = reinterpret_cast<float*>(dv + M);     // M
  float* xv = rhs + M;                               // M
  float* A = xv + M;                                 // packed lower triangle
  __shared__ float Blk[kSB][kSB + 1];                // staging of the current diagonal block
  __shared__ float Ld[kSB][kSB + 1];                 // padded diagonal factor of the current block
  __shared__ float rd[kSB];                          // its reciprocal pivots
  __shared__ double red[2][4];
  __shared__ double sc[4];
  const int tid = threadIdx.x;
  const int nt = blockDim.x;
  const int wave = tid >> 6, lane = tid & 63;
  const double Md = static_cast<double>(M);
  if (tid == 0) *info = 0;

  // 1. counts -> LDS (lower part; exact as floats below 2^24), row sums, trace
  double trl = 0.0, sgl = 0.0;
  if (has_random) {
    for (int64_t i = wave; i < M; i += nt / 64) {
      long long sum = 0;
      for (int64_t j0 = 0; j0 < M; j0 += 512) {
        int32_t v[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const int64_t j = j0 + q * 64 + lane;
          v[q] = C[i * M + (j < M ? j : 0)];
          v[q] = j < M ? v[q] : 0;
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const int64_t j = j0 + q * 64 + lane;
          sum += v[q];
          if (j <= i) A[tri(i, j)] = static_cast<float>(v[q]);
          trl += j == i ? static_cast<double>(v[q]) : 0.0;
        }
      }
      for (int off = 32; off > 0; off >>= 1) sum += __shfl_xor(sum, off);
      if (lane == 0) dv[i] = static_cast<double>(sum);
      sgl += lane == 0 ? static_cast<double>(sum) : 0.0;
    }
  }
  for (int off = 32; off > 0; off >>= 1) {
    trl += __shfl_xor(trl, off);
    sgl += __shfl_xor(sgl, off);
  }
  if (lane == 0) {
    red[0][wave] = trl;
    red[1][wave] = sgl;
  }
  __syncthreads();
  if (tid == 0) {
    double tr = 0.0, sg = 0.0;
    for (int w = 0; w < nt / 64; ++w) {
      tr += red[0][w];
      sg += red[1][w];
    }
    const double tr_pgp = alpha * (Md - 1.0) + 2.0 * wr * (tr - sg / Md);
    sc[0] = sg;
    sc[1] = tr_pgp / (Md - 1.0);
    sc[2] = static_cast<double>(fef[1]) - static_cast<double>(fef[0]);
  }
  __syncthreads();
  const double sigma = sc[0], gamma = sc[1], delta = sc[2];

  // 2. G~ = alpha P + 2 wr P C P + gamma 11^T/M, lower triangle in place
  for (int64_t i = 0, base = 0; i < M; base += i + 1, ++i) {
    for (int64_t j = tid; j <= i; j += nt) {
      double v = alpha * ((i == j ? 1.0 : 0.0) - 1.0 / Md) + gamma / Md;
      if (has_random) v += 2.0 * wr * (static_cast<double>(A[base + j]) - (dv[i] + dv[j]) / Md + sigma / (Md * Md));
      A[base + j] = static_cast<float>(v);
    }
  }
  __syncthreads();

  // 3. right-hand side P r from the partial sums (8 loads in flight per thread)
  double sl = 0.0;
  for (int64_t j = tid; j < M; j += nt) {
    double v = 0.0;
    for (int64_t c0 = 0; c0 < nch; c0 += 8) {
      double t[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) t[q] = part[(c0 + q < nch ? c0 + q : 0) * M + j];
#pragma unroll
      for (int q = 0; q < 8; ++q) v += c0 + q < nch ? t[q] : 0.0;
    }
    dv[j] = v;
    sl += v;
  }
  for (int off = 32; off > 0; off >>= 1) sl += __shfl_xor(sl, off);
  if (lane == 0) red[0][wave] = sl;
  __syncthreads();
  if (tid == 0) {
    double t = 0.0;
    for (int w = 0; w < nt / 64; ++w) t += red[0][w];
    sc[3] = t / Md;
  }
  __syncthreads();
  for (int64_t j = tid; j < M; j += nt) rhs[j] = static_cast<float>(dv[j] - sc[3]);
  __syncthreads();

  // 4. Cholesky, 32-wide blocks
  for (int64_t o = 0; o < M; o += kSB) {
    const int nbe = static_cast<int>(M - o < kSB ? M - o : kSB);
    for (int t = tid; t < kSB * kSB; t += nt) {      // padded block: identity past nbe
      const int r = t / kSB, c = t % kSB;
      Blk[r][c] = (r < nbe && c <= r) ? A[tri(o + r, o + c)] : (r == c ? 1.f : 0.f);
    }
    __syncthreads();
    if (wave == 0) {
      float a[kSB];
#pragma unroll
      for (int c = 0; c < kSB; ++c) a[c] = Blk[lane & (kSB - 1)][c];
      chol_regs<kSB>(a, o, info);
      if (lane < kSB) {
#pragma unroll
        for (int c = 0; c < kSB; ++c) Blk[lane][c] = a[c];
      }
    }
    __syncthreads();
    for (int t = tid; t < kSB * kSB; t += nt) {
      const int r = t / kSB, c = t % kSB;
      const float v = c <= r ? Blk[r][c] : 0.f;
      Ld[r][c] = v;
      if (c == r) rd[r] = 1.0f / v;
      if (r < nbe && c <= r) A[tri(o + r, o + c)] = v;
    }
    __syncthreads();
    // rows below exist only when the diagonal block is full (nbe == kSB)
    const int64_t r0 = o + nbe;
    const int64_t T = M - r0;
    for (int64_t i = r0 + tid; i < M; i += nt) {
      float x[kSB];
      const int64_t bi = tri(i, o);
#pragma unroll
      for (int c = 0; c < kSB; ++c) x[c] = A[bi + c];
#pragma unroll
      for (int c = 0; c < kSB; ++c) {
        x[c] *= rd[c];
#pragma unroll
        for (int q = c + 1; q < kSB; ++q) x[q] -= x[c] * Ld[q][c];
        __builtin_amdgcn_sched_barrier(0);   // column by column: keeps register pressure low
      }
#pragma unroll
      for (int c = 0; c < kSB; ++c)
        A[bi + c] = x[c];
    }
    __syncthreads();
    const int64_t T4 = (T + 3) / 4;
    for (int64_t t = tid; t < T4 * T4; t += nt) {
      const int64_t I = t / T4, J = t % T4;
      if (J > I) continue;
      float acc[4][4] = {};
      int64_t pi[4], pj[4];
      bool oi[4], oj[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int64_t ri = r0 + 4 * I + q, rj = r0 + 4 * J + q;
        oi[q] = ri < M;
        oj[q] = rj < M;
        pi[q] = oi[q] ? tri(ri, o) : 0;
        pj[q] = oj[q] ? tri(rj, o) : 0;
      }
      for (int c = 0; c < nbe; ++c) {
        float pa[4], pb[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          pa[q] = oi[q] ? A[pi[q] + c] : 0.f;
          pb[q] = oj[q] ? A[pj[q] + c] : 0.f;
        }
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
          for (int r = 0; r < 4; ++r) acc[q][r] += pa[q] * pb[r];
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int64_t i = r0 + 4 * I + q;
        if (i >= M) continue;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t j = r0 + 4 * J + r;
          if (j <= i) A[tri(i, j)] -= acc[q][r];
        }
      }
    }
    __syncthreads();
  }

  // 5. forward substitution L x = rhs (one wavefront per diagonal block)
  for (int64_t o = 0; o < M; o += kSB) {
    const int nbe = static_cast<int>(M - o < kSB ? M - o : kSB);
    // strictly lower part of the diagonal block and its reciprocal pivots
    for (int t = tid; t < kSB * kSB; t += nt) {
      const int r = t / kSB, c = t % kSB;
      Blk[r][c] = (r < nbe && c < r) ? A[tri(o + r, o + c)] : 0.f;
      if (c == r) rd[r] = r < nbe ? 1.0f / A[tri(o + r, o + r)] : 1.f;
    }
    __syncthreads();
    if (wave == 0) {
      // b_k is final once the columns before k are applied: x_k = b_k / L_kk
      const int rl = lane & (kSB - 1);
      float b = lane < nbe ? rhs[o + lane] : 0.f;
      float lr[kSB];
#pragma unroll
      for (int c = 0; c < kSB; ++c) lr[c] = Blk[rl][c];
#pragma unroll
      for (int k = 0; k < kSB; ++k) b -= lr[k] * (bcast(b, k) * rd[k]);
      if (lane < nbe) xv[o + lane] = b * rd[rl];
    }
    __syncthreads();
    for (int64_t i = o + nbe + tid; i < M; i += nt) {
      float acc = 0.f;
      const int64_t bi = tri(i, o);
      for (int c = 0; c < nbe; ++c) acc += A[bi + c] * xv[o + c];
      rhs[i] -= acc;
    }
    __syncthreads();
  }

  // 6. backward substitution L^T z = x (z overwrites rhs)
  for (int64_t o = ((M - 1) / kSB) * kSB; o >= 0; o -= kSB) {
    const int nbe = static_cast<int>(M - o < kSB ? M - o : kSB);
    // Blk[r][k] = L[o+k][o+r] for k > r (the strictly upper part of L_jj^T)
    for (int t = tid; t < kSB * kSB; t += nt) {
      const int r = t / kSB, k = t % kSB;
      Blk[r][k] = (k < nbe && r < k) ? A[tri(o + k, o + r)] : 0.f;
      if (k == r) rd[r] = r < nbe ? 1.0f / A[tri(o + r, o + r)] : 1.f;
    }
    __syncthreads();
    if (wave == 0) {
      const int rl = lane & (kSB - 1);
      float b = lane < nbe ? xv[o + lane] : 0.f;
      float lc[kSB];
#pragma unroll
      for (int k = 0; k < kSB; ++k) lc[k] = Blk[rl][k];
#pragma unroll
      for (int k = kSB - 1; k >= 0; --k) b -= lc[k] * (bcast(b, k) * rd[k]);
      if (lane < nbe) rhs[o + lane] = b * rd[rl];
    }
    __syncthreads();
    for (int64_t i = tid; i < o; i += nt) {
      float acc = 0.f;
      for (int c = 0; c < nbe; ++c) acc += A[tri(o + c, i)] * rhs[o + c];
      xv[i] -= acc;
    }
    __syncthreads();
  }

  // 7. phi = Delta/M + psi
  for (int64_t i = tid; i < M; i += nt) phi[i] = static_cast<float>(delta / Md + static_cast<double>(rhs[i]));
}

__global__ void k_zero_info(int32_t* info) { *info = 0; }

// Multi-block path, diagonal block jb: one wavefront factors it in registers,
// writes L_jj back (zeros above the diagonal) and the padded factor with its
// reciprocal pivots to Ld for the panel kernel.
__global__ void __launch_bounds__(64) k_potrf(float* G, int64_t M, int64_t jb, int32_t* info, float* Ld) {
  const int64_t o = jb * kNB;
  const int n = static_cast<int>(M - o < kNB ? M - o : kNB);
  const int lane = threadIdx.x;
  const bool own = lane < n;
  float a[kNB];
#pragma unroll
  for (int c = 0; c < kNB; ++c) {
    const bool real = own && c < n && c <= lane;
    const float v = G[real ? (o + lane) * M + o + c : 0];
    a[c] = real ? v : (c == lane ? 1.f : 0.f);
  }
  chol_regs<kNB>(a, o, info);
#pragma unroll
  for (int c = 0; c < kNB; ++c) Ld[lane * kNB + c] = c <= lane ? a[c] : 0.f;
  Ld[kNB * kNB + lane] = 1.0f / lane_entry(a);
  if (own) {
#pragma unroll
    for (int c = 0; c < kNB; ++c)
      if (c < n) G[(o + lane) * M + o + c] = c <= lane ? a[c] : 0.f;
  }
}

// Panel: rows below block jb, X <- X L_jj^-T, one thread per row, right-looking.
__global__ void __launch_bounds__(256) k_trsm(float* G, int64_t M, int64_t jb, const float* __restrict__ Ld) {
  __shared__ float L[kNB][kNB + 1];
  __shared__ float rd[kNB];
  const int64_t o = jb * kNB;
  const int tid = threadIdx.x;
  for (int t = tid; t < kNB * kNB; t += 256) L[t / kNB][t % kNB] = Ld[t];
  if (tid < kNB) rd[tid] = Ld[kNB * kNB + tid];
  __syncthreads();
  const int64_t r = o + kNB + static_cast<int64_t>(blockIdx.x) * 256 + tid;
  if (r >= M) return;
  float x[kNB];
  float* row = G + r * M + o;
#pragma unroll
  for (int c = 0; c < kNB; ++c) x[c] = row[c];
#pragma unroll
  for (int c = 0; c < kNB; ++c) {
    x[c] *= rd[c];
#pragma unroll
    for (int q = c + 1; q < kNB; ++q) x[q] -= x[c] * L[q][c];
    __builtin_amdgcn_sched_barrier(0);
  }
#pragma unroll
  for (int c = 0; c < kNB; ++c) row[c] = x[c];
}

// Trailing update of tile (ib, kb), jb < kb <= ib: A_ib,kb -= L_ib,jb L_kb,jb^T.
__global__ void __launch_bounds__(256) k_syrk(float* G, int64_t M, int64_t jb) {
  const int64_t ib = jb + 1 + blockIdx.y, kb = jb + 1 + blockIdx.x;
  if (kb > ib) return;
  __shared__ float As[16][64 + 4];
  __shared__ float Bs[16][64 + 4];
  const int tid = threadIdx.x;
  const int ty = tid / 16, tx = tid % 16;
  const int64_t o = jb * kNB;
  const int n = static_cast<int>(M - o < kNB ? M - o : kNB);
  float acc[4][4] = {};
  for (int k0 = 0; k0 < n; k0 += 16) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int idx = tid + q * 256;
      const int r = idx / 16, kk = idx % 16;
      const int64_t gi = ib * kNB + r, gk = kb * kNB + r;
      const bool kin = k0 + kk < n;
      As[kk][r] = (kin && gi < M) ? G[gi * M + o + k0 + kk] : 0.f;
      Bs[kk][r] = (kin && gk < M) ? G[gk * M + o + k0 + kk] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        a[q] = As[kk][ty * 4 + q];
        b[q] = Bs[kk][tx * 4 + q];
      }
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[q][r] += a[q] * b[r];
    }
    __syncthreads();
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int64_t i = ib * kNB + ty * 4 + q;
    if (i >= M) continue;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t j = kb * kNB + tx * 4 + r;
      if (j < M && j <= i) G[i * M + j] -= acc[q][r];
    }
  }
}

// Multi-block path, triangular solves by segments [s0, s1) of at most kSeg
// rows: one workgroup substitutes inside a segment (64-row blocks, one
// wavefront per diagonal block); multi-block GEMVs carry a segment's
// contribution to the rows outside it.
constexpr int64_t kSeg = 2048;

// Forward: x[s0:s1) = L[s0:s1, s0:s1)^-1 rhs[s0:s1) (rhs holds the earlier segments' updates).
__global__ void __launch_bounds__(1024) k_trsv_fwd(const float* __restrict__ G, int64_t M, int64_t s0, int64_t s1,
                                                   float* __restrict__ rhs, float* __restrict__ x) {
  __shared__ float Blk[kNB][kNB + 1];
  __shared__ float rd[kNB];
  const int tid = threadIdx.x, nt = blockDim.x;
  const int wave = tid >> 6, lane = tid & 63;
  for (int64_t o = s0; o < s1; o += kNB) {
    const int nbe = static_cast<int>(s1 - o < kNB ? s1 - o : kNB);
    for (int t = tid; t < kNB * kNB; t += nt) {      // strictly lower part of L_jj
      const int r = t / kNB, c = t % kNB;
      Blk[r][c] = (r < nbe && c < r) ? G[(o + r) * M + o + c] : 0.f;
      if (c == r) rd[r] = r < nbe ? 1.0f / G[(o + r) * M + o + r] : 1.f;
    }
    __syncthreads();
    if (wave == 0) {
      float b = lane < nbe ? rhs[o + lane] : 0.f;
      float lr[kNB];
#pragma unroll
      for (int c = 0; c < kNB; ++c) lr[c] = Blk[lane][c];
#pragma unroll
      for (int k = 0; k < kNB; ++k) b -= lr[k] * (bcast(b, k) * rd[k]);
      if (lane < nbe) x[o + lane] = b * rd[lane];
    }
    __syncthreads();
    for (int64_t i = o + nbe + tid; i < s1; i += nt) {
      float acc = 0.f;
      const float* row = G + i * M + o;
#pragma unroll 8
      for (int c = 0; c < nbe; ++c) acc += row[c] * x[o + c];
      rhs[i] -= acc;
    }
    __syncthreads();
  }
}

// rhs[i] -= L[i, s0:s1) x[s0:s1) for i >= s1; one wavefront per row.
__global__ void __launch_bounds__(256) k_gemv_fwd(const float* __restrict__ G, int64_t M, int64_t s0, int64_t s1,
                                                  const float* __restrict__ x, float* __restrict__ rhs) {
  const int lane = threadIdx.x & 63;
  const int64_t i = s1 + ((static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) >> 6);
  if (i >= M) return;
  float acc = 0.f;
  for (int64_t c = s0 + lane; c < s1; c += 64) acc += G[i * M + c] * x[c];
  for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  if (lane == 0) rhs[i] -= acc;
}

// Backward: z[s0:s1) = L[s0:s1, s0:s1)^-T x[s0:s1) into rhs (x holds the later segments' updates).
__global__ void __launch_bounds__(1024) k_trsv_bwd(const float* __restrict__ G, int64_t M, int64_t s0, int64_t s1,
                                                   float* __restrict__ x, float* __restrict__ rhs) {
  __shared__ float Blk[kNB][kNB + 1];
  __shared__ float rd[kNB];
  const int tid = threadIdx.x, nt = blockDim.x;
  const int wave = tid >> 6, lane = tid & 63;
  for (int64_t o = s0 + ((s1 - s0 - 1) / kNB) * kNB; o >= s0; o -= kNB) {
    const int nbe = static_cast<int>(s1 - o < kNB ? s1 - o : kNB);
    for (int t = tid; t < kNB * kNB; t += nt) {      // Blk[r][k] = L[o+k][o+r], k > r
      const int r = t / kNB, k = t % kNB;
      Blk[r][k] = (k < nbe && r < k) ? G[(o + k) * M + o + r] : 0.f;
      if (k == r) rd[r] = r < nbe ? 1.0f / G[(o + r) * M + o + r] : 1.f;
    }
    __syncthreads();
    if (wave == 0) {
      float b = lane < nbe ? x[o + lane] : 0.f;
      float lc[kNB];
#pragma unroll
      for (int k = 0; k < kNB; ++k) lc[k] = Blk[lane][k];
#pragma unroll
      for (int k = kNB - 1; k >= 0; --k) b -= lc[k] * (bcast(b, k) * rd[k]);
      if (lane < nbe) rhs[o + lane] = b * rd[lane];
    }
    __syncthreads();
    for (int64_t i = s0 + tid; i < o; i += nt) {
      float acc = 0.f;
#pragma unroll 8
      for (int c = 0; c < nbe; ++c) acc += G[(o + c) * M + i] * rhs[o + c];
      x[i] -= acc;
    }
    __syncthreads();
  }
}

// x[i] -= sum_{c in [s0, s1)} L[c, i] z[c] for i < s0; one thread per row (coalesced over i).
__global__ void __launch_bounds__(256) k_gemv_bwd(const float* __restrict__ G, int64_t M, int64_t s0, int64_t s1,
                                                  const float* __restrict__ z, float* __restrict__ x) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= s0) return;
  float acc = 0.f;
  for (int64_t c = s0; c < s1; ++c) acc += G[c * M + i] * z[c];
  x[i] -= acc;
}

__global__ void k_finish(const float* __restrict__ z, int64_t M, const double* __restrict__ scal,
                         float* __restrict__ phi) {
  const double base = scal[3] / static_cast<double>(M);
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < M;
       i += static_cast<int64_t>(gridDim.x) * blockDim.x)
    phi[i] = static_cast<float>(base + static_cast<double>(z[i]));
}

int check_plan(const gnnshap_sample_plan* p, const gnnshap_class* classes) {
  if (!p) return gnnshap::fail(GNNSHAP_EINVAL, "plan is NULL");
  if (p->num_players < 2 || p->num_rows < 2 || (p->num_rows % 2) ||
      p->words_per_row != (p->num_players + 63) / 64 || p->num_classes < 1 || p->random_begin < 0 ||
      p->random_begin > p->num_rows / 2)
    return gnnshap::fail(GNNSHAP_EINVAL, "plan is not the output of gnnshap_plan_samples");
  if (classes) {
    int64_t row = 0;
    for (int64_t i = 0; i < p->num_classes; ++i) {
      if (classes[i].row_begin != row || classes[i].row_count < 1 ||
          (classes[i].full != 0) != (row < p->random_begin))
        return gnnshap::fail(GNNSHAP_EINVAL, "class table inconsistent at record %lld", (long long)i);
      if (!classes[i].full && classes[i].weight != p->random_weight)
        return gnnshap::fail(GNNSHAP_EINVAL, "random rows must share the plan's random weight");
      row += classes[i].row_count;
    }
    if (row != p->num_rows / 2) return gnnshap::fail(GNNSHAP_EINVAL, "class table does not cover k/2 rows");
  }
  return GNNSHAP_OK;
}

// C(n, r) in fp64 (exact while below 2^53; the enumerated classes stay far below).
double binom_d(int64_t n, int64_t r) {
  if (r < 0 || r > n) return 0.0;
  if (r > n - r) r = n - r;
  double v = 1.0;
  for (int64_t i = 1; i <= r; ++i) v = v * static_cast<double>(n - r + i) / static_cast<double>(i);
  return v;
}

}  // namespace

extern "C" int gnnshap_solve_workspace(const gnnshap_sample_plan* plan, size_t* bytes) {
  gnnshap::clear_error();
  if (!bytes) return gnnshap::fail(GNNSHAP_EINVAL, "bytes is NULL");
  if (int st = check_plan(plan, nullptr)) return st;
  gnnshap::Carver c(nullptr);
  carve(c, plan);
  *bytes = c.bytes();
  return GNNSHAP_OK;
}

extern "C" int gnnshap_solve_wls(const gnnshap_sample_plan* plan, const gnnshap_class* classes,
                                 const uint64_t* masks, const float* y, const float* f_empty_full, float* phi,
                                 int32_t* info, void* ws, size_t ws_bytes, void* stream) {
  GS_TRY_BEGIN
  gnnshap::clear_error();
  if (!classes || !masks || !y || !f_empty_full || !phi || !info || !ws)
    return gnnshap::fail(GNNSHAP_EINVAL, "null argument");
  if (int st = check_plan(plan, classes)) return st;
  gnnshap::Carver need(nullptr);
  carve(need, plan);
  if (ws_bytes < need.bytes()) return gnnshap::fail(GNNSHAP_ECAPACITY, "solve workspace needs %zu bytes", need.bytes());
  gnnshap::Carver cv(ws);
  const Ws w = carve(cv, plan);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t M = plan->num_players;
  const int64_t wpr = plan->words_per_row;
  const int64_t half = plan->num_rows / 2;
  const int64_t rb0 = plan->random_begin;
  const int64_t kr = half - rb0;
  const bool has_random = kr > 0;
  const double wr = has_random ? plan->random_weight : 0.0;
  // Enumerated classes: P (sum over the class and its complements) P = w kappa C(M-2, c-1) P.
  double alpha = 0.0;
  for (int64_t i = 0; i < plan->num_classes; ++i) {
    if (!classes[i].full) continue;
    const int64_t c = classes[i].size;
    const double kappa = 2 * c < M ? 2.0 : 1.0;
    alpha += classes[i].weight * kappa * binom_d(M - 2, c - 1);
  }
  GS_HIP(hipMemcpyAsync(w.classes, classes, plan->num_classes * sizeof(gnnshap_class), hipMemcpyHostToDevice, s));
  int32_t* counts = reinterpret_cast<int32_t*>(w.G);
  if (has_random) {
    const int64_t nrb = gnnshap::ceil_div(kr, 64);
    {
      GS_TIMED("k_transpose", s);
      k_transpose<<<dim3(static_cast<unsigned>(nrb), static_cast<unsigned>(wpr)), 64, 0, s>>>(masks, wpr, rb0, kr, M, w.T);
    }
    GS_LAUNCHED();
    const unsigned nb = static_cast<unsigned>(gnnshap::ceil_div(M, 64));
    {
      GS_TIMED("k_gram", s);
      k_gram<<<dim3(nb, nb), 256, 0, s>>>(w.T, nrb, M, counts);
    }
    GS_LAUNCHED();
  }
  const int64_t nch = n_chunks(half);
  const int64_t rpc = gnnshap::ceil_div(half, nch);
  {
    GS_TIMED("k_rhs_part", s);
    k_rhs_part<<<static_cast<unsigned>(nch), 256, 0, s>>>(masks, wpr, half, M, y, w.classes, plan->num_classes,
                                                           f_empty_full, rpc, w.part);
  }
  GS_LAUNCHED();

  const size_t small_bytes = small_lds_bytes(M);
  if (small_bytes <= static_cast<size_t>(gnnshap::max_lds_bytes())) {
    bool ok = small_bytes <= 65536;
    if (!ok) {
      ok = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_solve_small), hipFuncAttributeMaxDynamicSharedMemorySize,
                               static_cast<int>(small_bytes)) == hipSuccess;
      (void)hipGetLastError();
    }
    if (ok) {
      {
        GS_TIMED("k_solve_small", s);
        k_solve_small<<<1, 256, small_bytes, s>>>(counts, M, has_random, alpha, wr, f_empty_full, w.part, nch, info,
                                                  phi);
      }
      GS_LAUNCHED();
      return GNNSHAP_OK;
    }
  }

  k_zero_info<<<1, 1, 0, s>>>(info);
  GS_LAUNCHED();
  if (has_random) {
    k_rowsum<<<static_cast<unsigned>(gnnshap::ceil_div(M * 64, 256)), 256, 0, s>>>(counts, M, w.usum);
    GS_LAUNCHED();
  }
  k_scalars<<<1, 256, 0, s>>>(counts, w.usum, M, has_random, alpha, wr, f_empty_full, w.scal);
  GS_LAUNCHED();
  k_build<<<gnnshap::grid_for(M * M, 256, 16384), 256, 0, s>>>(w.G, w.usum, M, has_random, alpha, wr, w.scal);
  GS_LAUNCHED();
  k_rhs_finish<<<1, 1024, 0, s>>>(w.part, nch, M, w.rhs, w.scal);
  GS_LAUNCHED();
  const int64_t nblk = gnnshap::ceil_div(M, kNB);
  for (int64_t jb = 0; jb < nblk; ++jb) {
    {
      GS_TIMED("k_potrf", s);
      k_potrf<<<1, 64, 0, s>>>(w.G, M, jb, info, w.Ld);
    }
    GS_LAUNCHED();
    const int64_t rest = nblk - jb - 1;
    if (rest > 0) {
      const int64_t rows = M - (jb + 1) * kNB;
      {
        GS_TIMED("k_trsm", s);
        k_trsm<<<static_cast<unsigned>(gnnshap::ceil_div(rows, 256)), 256, 0, s>>>(w.G, M, jb, w.Ld);
      }
      GS_LAUNCHED();
      {
        GS_TIMED("k_syrk", s);
        k_syrk<<<dim3(static_cast<unsigned>(rest), static_cast<unsigned>(rest)), 256, 0, s>>>(w.G, M, jb);
      }
      GS_LAUNCHED();
    }
  }
  // L x = rhs, L^T psi = x (psi into rhs), phi = Delta/M + psi
  for (int64_t s0 = 0; s0 < M; s0 += kSeg) {
    const int64_t s1 = std::min(M, s0 + kSeg);
    {
      GS_TIMED("k_trsv", s);
      k_trsv_fwd<<<1, 1024, 0, s>>>(w.G, M, s0, s1, w.rhs, w.x);
    }
    GS_LAUNCHED();
    if (s1 < M) {
      k_gemv_fwd<<<static_cast<unsigned>(gnnshap::ceil_div((M - s1) * 64, 256)), 256, 0, s>>>(w.G, M, s0, s1, w.x,
                                                                                             w.rhs);
      GS_LAUNCHED();
    }
  }
  for (int64_t s0 = ((M - 1) / kSeg) * kSeg; s0 >= 0; s0 -= kSeg) {
    const int64_t s1 = std::min(M, s0 + kSeg);
    {
      GS_TIMED("k_trsv", s);
      k_trsv_bwd<<<1, 1024, 0, s>>>(w.G, M, s0, s1, w.x, w.rhs);
    }
    GS_LAUNCHED();
    if (s0 > 0) {
      k_gemv_bwd<<<static_cast<unsigned>(gnnshap::ceil_div(s0, 256)), 256, 0, s>>>(w.G, M, s0, s1, w.rhs, w.x);
      GS_LAUNCHED();
    }
  }
  k_finish<<<gnnshap::grid_for(M, 256, 1024), 256, 0, s>>>(w.rhs, M, w.scal, phi);
  GS_LAUNCHED();
  return GNNSHAP_OK;
  GS_TRY_END
}
