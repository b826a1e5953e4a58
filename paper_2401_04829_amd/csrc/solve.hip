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
// Systems of up to 448 players are factored and solved by one workgroup
// (several targets' systems side by side in a batch).  Larger ones, up to
// the iterative threshold (above it the system is not formed: cg.hip), use a
// blocked right-looking Cholesky over the whole GPU with 128-wide panels: one workgroup factors the diagonal block and
// inverts its factor, then the panel solve (a product with that inverse) and
// the trailing update run as fp32 MFMA GEMMs.  The triangular solves go by
// 256-row segments whose triangle sits in LDS, with multi-block GEMVs carrying
// each segment to the rows outside it.  The right-hand side is accumulated in
// fp64.
#include <algorithm>
#include <cmath>

#include "batch.h"
#include "cg.h"
#include "nibble.h"
#include "common.h"

namespace {

constexpr int kPB = 128;       // panel width, multi-block Cholesky
constexpr int kTB = 64;        // diagonal block of the triangular solves (one wavefront)
constexpr int64_t kSeg = 256;  // segment of the triangular solves (its triangle in LDS)
constexpr int kMaxChunks = 256;
constexpr int kMidMax = 448;   // largest system of the global-memory one-workgroup path
constexpr int64_t kPanelMin = 192;  // larger systems (up to kMidMax) take the panel path

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

struct Ws {
  gnnshap_class* classes;
  uint64_t* T;       // nrb x M: bit b of T[rb, j] = player j in random row rb*64+b
  float* G;          // M rows of ld floats (int32 counts first, then the system, lower part factored)
  int64_t* usum;     // M: row sums of the counts
  double* scal;      // [0] trace, [1] sigma, [2] gamma, [3] delta, [4] f0
  double* dz;        // half: z_b - z_{b+half}
  double* part;      // nch x M partial right-hand sides
  double* dv;        // M: summed right-hand side before centring
  double* bsum;      // per-block sums of dv
  float* rhs;        // M
  float* x;          // M
  float* Winv;       // kPB x kPB inverse of the current diagonal factor
  float* Wd;         // one-workgroup mid-size path: ceil(M/64) inverse diagonal factors (64 x 64)
  gnnshap::CgWs cg;  // iterative path only (no G, Winv, Wd)
};

// Systems above the plan's threshold are solved iteratively (Sec. 3.5).
bool iterative(const gnnshap_sample_plan* p) { return p->num_players > gnnshap::iterative_threshold(p); }

// The iterative solver's shape for a plan and its class table; without a
// table (workspace queries), for the table gnnshap_plan_samples gives the plan.
gnnshap::CgShape cg_shape_of(const gnnshap_sample_plan* p, const gnnshap_class* classes = nullptr) {
  const int64_t kr = p->num_rows / 2 - p->random_begin;
  if (classes)
    return gnnshap::cg_shape(p->num_players, p->words_per_row, kr, p->random_begin, classes, p->num_classes);
  gnnshap_sample_plan q = *p;
  std::vector<gnnshap_class> tab(static_cast<size_t>(std::max<int64_t>(p->num_classes, 1)));
  if (gnnshap_plan_samples(&q, tab.data(), static_cast<int64_t>(tab.size())) != GNNSHAP_OK ||
      q.num_rows != p->num_rows || q.random_begin != p->random_begin || q.num_classes != p->num_classes) {
    gnnshap::clear_error();
    return gnnshap::cg_shape(p->num_players, p->words_per_row, kr, p->random_begin, nullptr, 0);
  }
  return gnnshap::cg_shape(p->num_players, p->words_per_row, kr, p->random_begin, tab.data(), q.num_classes);
}

// Row stride of G: a multiple of 64 floats keeps every row 256-byte aligned.
int64_t ld_of(int64_t M) { return gnnshap::ceil_div(M, 64) * 64; }

// Row chunks of the right-hand side: enough wavefronts (word columns x chunks,
// about 32768) that each one's chain of row loads is short, at least 64 rows
// per chunk.
int64_t n_chunks(int64_t half, int64_t wpr) {
  int64_t c = gnnshap::ceil_div(32768, wpr);
  const int64_t by_rows = gnnshap::ceil_div(half, 64);
  if (c > by_rows) c = by_rows;
  if (c > kMaxChunks) c = kMaxChunks;
  return c < 1 ? 1 : c;
}

// Row chunks of the chunked right-hand side (systems of at most kMidMax players).
constexpr int kTileRows = 256;
constexpr int kTileWords = (kMidMax + 63) / 64;          // mask words per row at most
constexpr int kTileClasses = 256;                         // classes of a system of <= kMidMax players

int64_t tile_chunks(int64_t half) { return gnnshap::ceil_div(half, kTileRows); }

// Iterative path: row chunks of the right-hand side's enumerated rows (from
// the row-major masks) and of its random rows (kTabWords row blocks of the
// bit-transposed rows each).
int64_t rhs_enum_chunks(const gnnshap_sample_plan* p) {
  return p->random_begin > 0 ? n_chunks(p->random_begin, p->words_per_row) : 0;
}
int64_t rhs_rand_chunks(const gnnshap_sample_plan* p) {
  const int64_t kr = p->num_rows / 2 - p->random_begin;
  return gnnshap::ceil_div(gnnshap::ceil_div(kr, 64), gnnshap::kTabWords);
}

Ws carve(gnnshap::Carver& c, const gnnshap_sample_plan* p, const gnnshap_class* classes = nullptr) {
  Ws w;
  const int64_t M = p->num_players;
  const int64_t half = p->num_rows / 2;
  const int64_t kr = half - p->random_begin;
  const int64_t nrb = gnnshap::ceil_div(kr, 64);
  w.classes = c.take<gnnshap_class>(p->num_classes > 0 ? p->num_classes : 1);
  w.T = c.take<uint64_t>((nrb > 0 ? nrb : 1) * M);
  if (iterative(p)) {
    w.G = nullptr;
    w.usum = nullptr;
    w.scal = nullptr;
    w.dz = c.take<double>(half);
    w.part = c.take<double>(std::max<int64_t>(rhs_enum_chunks(p) + rhs_rand_chunks(p), 1) * M);
    w.dv = c.take<double>(M);
    w.bsum = c.take<double>(gnnshap::ceil_div(M, 256));
    w.rhs = w.x = w.Winv = w.Wd = nullptr;
    w.cg = gnnshap::cg_carve(c, cg_shape_of(p, classes));
    return w;
  }
  w.cg = gnnshap::CgWs{};
  w.G = c.take<float>(M * ld_of(M));
  w.usum = c.take<int64_t>(M);
  w.scal = c.take<double>(16);
  w.dz = c.take<double>(half);
  w.part = c.take<double>(std::max(n_chunks(half, p->words_per_row), tile_chunks(half)) * M);
  w.dv = c.take<double>(M);
  w.bsum = c.take<double>(gnnshap::ceil_div(M, 256));
  w.rhs = c.take<float>(M);
  w.x = c.take<float>(M);
  w.Winv = c.take<float>(kPB * kPB);
  w.Wd = c.take<float>(M <= kMidMax ? gnnshap::ceil_div(M, 64) * 64 * 64 : 1);
  return w;
}

__device__ __forceinline__ float bcast(float v, int lane) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  return v;
}

// One stage of the 64 x 64 bit-matrix transpose across a wavefront: lanes l
// and l ^ S exchange S x S bit blocks (m selects the low S bits of every
// 2S-bit group).
template <int S>
__device__ __forceinline__ uint64_t transpose_stage(uint64_t x, int lane, uint64_t m) {
  const uint64_t p = __shfl_xor(static_cast<unsigned long long>(x), S);
  return (lane & S) ? (((p >> S) & m) | (x & ~m)) : ((x & m) | ((p & m) << S));
}

// T[rb, j]: transpose 64 rows x 64 players, lane = row in, lane = player out,
// in six exchange stages (blocks of 32, 16, ..., 1 bits).  One wave per (rb, word).
__device__ __forceinline__ void transpose_body(const uint64_t* __restrict__ masks, int64_t wpr, int64_t row0,
                                               int64_t nrows, int64_t M, uint64_t* __restrict__ T, int64_t rb,
                                               int64_t w) {
  const int lane = threadIdx.x & 63;
  const int64_t r = rb * 64 + lane;
  uint64_t x = r < nrows ? masks[(row0 + r) * wpr + w] : 0;
  x = transpose_stage<32>(x, lane, 0x00000000FFFFFFFFull);
  x = transpose_stage<16>(x, lane, 0x0000FFFF0000FFFFull);
  x = transpose_stage<8>(x, lane, 0x00FF00FF00FF00FFull);
  x = transpose_stage<4>(x, lane, 0x0F0F0F0F0F0F0F0Full);
  x = transpose_stage<2>(x, lane, 0x3333333333333333ull);
  x = transpose_stage<1>(x, lane, 0x5555555555555555ull);
  const int64_t j = w * 64 + lane;
  if (j < M) T[rb * M + j] = x;
}

__global__ void __launch_bounds__(64) k_transpose(const uint64_t* __restrict__ masks, int64_t wpr, int64_t row0,
                                                  int64_t nrows, int64_t M, uint64_t* __restrict__ T) {
  transpose_body(masks, wpr, row0, nrows, M, T, blockIdx.x, blockIdx.y);
}

// T as above, and the same words in row blocks: B[(rb * wpr + w) * 64 + b] =
// word w of row rb * 64 + b (zero beyond nrows), so that a wave reading word
// w of 64 consecutive rows reads 512 contiguous bytes.
// Workgroup (rb, y): wavefront w' handles word column w = 8 y + w' of row
// block rb, so the eight wavefronts read neighbouring words of the same 64
// rows (whole cache lines per workgroup) and write 8 x 512 contiguous bytes
// of each copy.
__global__ void __launch_bounds__(512) k_transpose_blocked(const uint64_t* __restrict__ masks, int64_t wpr,
                                                           int64_t row0, int64_t nrows, int64_t M,
                                                           uint64_t* __restrict__ T, uint64_t* __restrict__ B) {
  const int64_t rb = blockIdx.x;
  const int64_t w = static_cast<int64_t>(blockIdx.y) * 8 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (w >= wpr) return;
  const int lane = threadIdx.x & 63;
  const int64_t r = rb * 64 + lane;
  B[(rb * wpr + w) * 64 + lane] = r < nrows ? masks[(row0 + r) * wpr + w] : 0;
  transpose_body(masks, wpr, row0, nrows, M, T, rb, w);
}

// Counts C[i, j] = sum_rb popcount(T[rb, i] & T[rb, j]) for 64x64 tiles with J >= I,
// stored in both halves (row stride ld).
// Row sums of a 64 x 64 count tile (I, J) held 4 x 4 per thread (thread
// (ty, tx) = (tid / 16, tid % 16) holds rows ty + 16 q and columns tx + 16 r,
// q, r < 4, so that a wavefront's LDS reads of the tile's words fall on
// consecutive words: no bank conflicts),
// added to usum with integer atomics (exact in any order): rows of I get the
// tile's row sums; for an off-diagonal tile the rows of J get its column
// sums (the mirrored tile).  Every thread of the workgroup calls it.
__device__ __forceinline__ void tile_row_sums(const int (&acc)[4][4], int64_t M, int64_t I, int64_t J,
                                              int64_t* __restrict__ usum) {
  __shared__ int colsum[64];
  const int tid = threadIdx.x, ty = tid / 16, tx = tid % 16;
  if (tid < 64) colsum[tid] = 0;
  __syncthreads();
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    int rs = acc[q][0] + acc[q][1] + acc[q][2] + acc[q][3];
#pragma unroll
    for (int off = 8; off > 0; off >>= 1) rs += __shfl_xor(rs, off, 16);
    const int64_t i = I * 64 + ty + 16 * q;
    if (tx == 0 && i < M && rs != 0) atomicAdd(reinterpret_cast<unsigned long long*>(&usum[i]),
                                                static_cast<unsigned long long>(rs));
  }
  if (I != J) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int cs = acc[0][r] + acc[1][r] + acc[2][r] + acc[3][r];
      if (cs != 0) atomicAdd(&colsum[tx + 16 * r], cs);
    }
    __syncthreads();
    const int64_t j = J * 64 + tid;
    if (tid < 64 && j < M && colsum[tid] != 0)
      atomicAdd(reinterpret_cast<unsigned long long*>(&usum[j]), static_cast<unsigned long long>(colsum[tid]));
  }
}

// usum: NULL, or row sums to add the tile's sums to (tile_row_sums).
__device__ __forceinline__ void gram_body(const uint64_t* __restrict__ T, int64_t nrb, int64_t M, int64_t ld,
                                          int32_t* __restrict__ C, int64_t I, int64_t J,
                                          int64_t* __restrict__ usum = nullptr) {
  if (J < I) return;
  __shared__ uint64_t Ti[16][64];
  __shared__ uint64_t Tj[16][64];
  const int tid = threadIdx.x;
  const int ty = tid / 16, tx = tid % 16;
  int acc[4][4] = {};
  // the next stage's words are fetched while the current stage is counted
  uint64_t ni[4], nj[4];
  auto fetch = [&](int64_t k0) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int idx = tid + q * 256;
      const int kk = idx / 64, c = idx % 64;
      const int64_t i = I * 64 + c, j = J * 64 + c;
      const bool kin = k0 + kk < nrb;
      ni[q] = (kin && i < M) ? T[(k0 + kk) * M + i] : 0;
      nj[q] = (kin && j < M) ? T[(k0 + kk) * M + j] : 0;
    }
  };
  fetch(0);
  for (int64_t k0 = 0; k0 < nrb; k0 += 16) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int idx = tid + q * 256;
      Ti[idx / 64][idx % 64] = ni[q];
      Tj[idx / 64][idx % 64] = nj[q];
    }
    __syncthreads();
    if (k0 + 16 < nrb) fetch(k0 + 16);
#pragma unroll 4
    for (int kk = 0; kk < 16; ++kk) {
      uint64_t a[4], b[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        a[q] = Ti[kk][ty + 16 * q];
        b[q] = Tj[kk][tx + 16 * q];
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
    const int64_t i = I * 64 + ty + 16 * q;
    if (i >= M) continue;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t j = J * 64 + tx + 16 * r;
      if (j >= M) continue;
      C[i * ld + j] = acc[q][r];
      C[j * ld + i] = acc[q][r];
    }
  }
  if (usum) tile_row_sums(acc, M, I, J, usum);
}

// The same counts over the row words [w0, w1) only, added to C with integer
// atomics (exact in any order; C starts at zero).  A diagonal tile adds each
// of its entries once, an off-diagonal tile adds both halves.
__device__ __forceinline__ void gram_part_body(const uint64_t* __restrict__ T, int64_t w0, int64_t w1, int64_t M,
                                               int64_t ld, int32_t* __restrict__ C, int64_t I, int64_t J,
                                               int64_t* __restrict__ usum) {
  __shared__ uint64_t Ti[16][64];
  __shared__ uint64_t Tj[16][64];
  const int tid = threadIdx.x;
  const int ty = tid / 16, tx = tid % 16;
  int acc[4][4] = {};
  uint64_t ni[4], nj[4];
  auto fetch = [&](int64_t k0) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int idx = tid + q * 256;
      const int kk = idx / 64, c = idx % 64;
      const int64_t i = I * 64 + c, j = J * 64 + c;
      const bool kin = k0 + kk < w1;
      ni[q] = (kin && i < M) ? T[(k0 + kk) * M + i] : 0;
      nj[q] = (kin && j < M) ? T[(k0 + kk) * M + j] : 0;
    }
  };
  fetch(w0);
  for (int64_t k0 = w0; k0 < w1; k0 += 16) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int idx = tid + q * 256;
      Ti[idx / 64][idx % 64] = ni[q];
      Tj[idx / 64][idx % 64] = nj[q];
    }
    __syncthreads();
    if (k0 + 16 < w1) fetch(k0 + 16);
#pragma unroll 4
    for (int kk = 0; kk < 16; ++kk) {
      uint64_t a[4], b[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        a[q] = Ti[kk][ty + 16 * q];
        b[q] = Tj[kk][tx + 16 * q];
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
    const int64_t i = I * 64 + ty + 16 * q;
    if (i >= M) continue;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t j = J * 64 + tx + 16 * r;
      if (j >= M || acc[q][r] == 0) continue;
      atomicAdd(&C[i * ld + j], acc[q][r]);
      if (I != J) atomicAdd(&C[j * ld + i], acc[q][r]);
    }
  }
  tile_row_sums(acc, M, I, J, usum);
}

__global__ void __launch_bounds__(256) k_gram(const uint64_t* __restrict__ T, int64_t nrb, int64_t M, int64_t ld,
                                              int32_t* __restrict__ C) {
  gram_body(T, nrb, M, ld, C, blockIdx.y, blockIdx.x);
}

// usum[i] = sum_j C[i, j]; one wave per row.
__global__ void __launch_bounds__(256) k_rowsum(const int32_t* __restrict__ C, int64_t M, int64_t ld,
                                                int64_t* __restrict__ usum) {
  const int lane = threadIdx.x & 63;
  const int64_t i = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) >> 6;
  if (i >= M) return;
  long long s = 0;
  for (int64_t j = lane; j < M; j += 64) s += C[i * ld + j];
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
  if (lane == 0) usum[i] = s;
}

// scal: trace and sigma of the counts (exact), gamma, Delta, f0.  One block.
__device__ __forceinline__ void scalars_body(const int32_t* __restrict__ C, const int64_t* __restrict__ usum,
                                             int64_t M, int64_t ld, bool has_random, double alpha, double wr,
                                             const float* __restrict__ fef, double* scal) {
  __shared__ long long st[256], ss[256];
  const int tid = threadIdx.x;
  long long tr = 0, sg = 0;
  if (has_random)
    for (int64_t i = tid; i < M; i += 256) {
      tr += C[i * ld + i];
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
    if (fef) {
      scal[3] = static_cast<double>(fef[1]) - static_cast<double>(fef[0]);
      scal[4] = static_cast<double>(fef[0]);
    }
  }
}

__global__ void __launch_bounds__(256) k_scalars(const int32_t* __restrict__ C, const int64_t* __restrict__ usum,
                                                 int64_t M, int64_t ld, bool has_random, double alpha, double wr,
                                                 const float* __restrict__ fef, double* scal) {
  scalars_body(C, usum, M, ld, has_random, alpha, wr, fef, scal);
}

// Row i of the lower triangle: counts (int32) -> G~ (fp32) in place.
// Entry (i, j) of G~ from the integer counts: base + alpha [i = j]
// + 2 wr (c_ij - (u_i + u_j)/M), in fp64, rounded once to fp32.  `Gb`
// holds the per-system constants (the build kernel and the panel path's
// loads use the same expression, so G~ has the same bits either way).
struct GtBuild {
  double base, alpha, wr2, inv_m;
  bool has_random;
};

__device__ __forceinline__ GtBuild gt_build(int64_t M, bool has_random, double alpha, double wr,
                                            const double* __restrict__ scal) {
  const double inv_m = 1.0 / static_cast<double>(M);
  const double sigma = scal[1], gamma = scal[2];
  GtBuild b;
  b.base = -alpha * inv_m + gamma * inv_m + (has_random ? 2.0 * wr * sigma * inv_m * inv_m : 0.0);
  b.alpha = alpha;
  b.wr2 = 2.0 * wr;
  b.inv_m = inv_m;
  b.has_random = has_random;
  return b;
}

__device__ __forceinline__ float gt_entry(const GtBuild& b, int32_t cij, int64_t ui, int64_t uj, bool diag) {
  double v = b.base + (diag ? b.alpha : 0.0);
  if (b.has_random) v += b.wr2 * (static_cast<double>(cij) - static_cast<double>(ui + uj) * b.inv_m);
  return static_cast<float>(v);
}

__device__ __forceinline__ void build_row(float* G, const int64_t* __restrict__ usum, int64_t M, int64_t ld,
                                          bool has_random, double alpha, double wr, const double* __restrict__ scal,
                                          int64_t i) {
  const GtBuild b = gt_build(M, has_random, alpha, wr, scal);
  for (int64_t j = threadIdx.x; j <= i; j += blockDim.x) {
    const int32_t cij = has_random ? reinterpret_cast<const int32_t*>(G)[i * ld + j] : 0;
    G[i * ld + j] = gt_entry(b, cij, has_random ? usum[i] : 0, has_random ? usum[j] : 0, i == j);
  }
}

// In place: counts (int32) -> G~ (fp32) on the lower triangle (the factorisation reads nothing else).
__global__ void __launch_bounds__(256) k_build(float* G, const int64_t* __restrict__ usum, int64_t M, int64_t ld,
                                               bool has_random, double alpha, double wr,
                                               const double* __restrict__ scal) {
  build_row(G, usum, M, ld, has_random, alpha, wr, scal, blockIdx.x);   // one block per row
}

// dz_b = z_b - z_{b+half}, z_b = w_b (y_b - f0 - Delta/M |S_b|) for b < half; a
// representative row has its class's size, its complement M minus that.
__device__ __forceinline__ void dz_body(const float* __restrict__ y, int64_t half, int64_t M,
                                        const gnnshap_class* __restrict__ cls, int64_t ncls,
                                        const float* __restrict__ fef, double* __restrict__ dz, int64_t b) {
  if (b >= half) return;
  const double Md = static_cast<double>(M);
  const double f0 = static_cast<double>(fef[0]);
  const double delta = static_cast<double>(fef[1]) - f0;
  int64_t lo = 0, hi = ncls - 1;
  while (lo < hi) {
    const int64_t mid = (lo + hi + 1) >> 1;
    if (cls[mid].row_begin <= b) lo = mid; else hi = mid - 1;
  }
  const double w = cls[lo].weight;
  const int64_t pc = cls[lo].size;
  const double z1 = w * (static_cast<double>(y[b]) - f0 - delta / Md * static_cast<double>(pc));
  const double z2 = w * (static_cast<double>(y[b + half]) - f0 - delta / Md * static_cast<double>(M - pc));
  dz[b] = z1 - z2;
}

__global__ void __launch_bounds__(256) k_dz(const float* __restrict__ y, int64_t half, int64_t M,
                                            const gnnshap_class* __restrict__ cls, int64_t ncls,
                                            const float* __restrict__ fef, double* __restrict__ dz) {
  dz_body(y, half, M, cls, ncls, fef, dz, static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x);
}

// Partial right-hand sides: part[ch, j] = sum_{b in chunk ch} dz_b m_bj.  A
// wavefront owns one 64-player word column and the rows of one chunk: each
// row's word and dz_b are wave-uniform (scalar loads) and every lane tests
// its own bit.
__device__ __forceinline__ void rhs_part_body(const uint64_t* __restrict__ masks, int64_t wpr, int64_t half,
                                              int64_t M, const double* __restrict__ dz, int64_t rows_per_chunk,
                                              double* __restrict__ part, int64_t bx, int64_t chunk) {
  const int lane = threadIdx.x & 63;
  const int64_t w = bx * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (w >= wpr) return;
  const int64_t r0 = chunk * rows_per_chunk;
  const int64_t r1 = r0 + rows_per_chunk < half ? r0 + rows_per_chunk : half;
  const uint64_t* col = masks + w;
  double acc = 0.0;
  int64_t b = r0;
  for (; b + 8 <= r1; b += 8) {
    uint64_t m[8];
    double d[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      m[q] = col[(b + q) * wpr];
      d[q] = dz[b + q];
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) acc += ((m[q] >> lane) & 1) ? d[q] : 0.0;
  }
  for (; b < r1; ++b) acc += ((col[b * wpr] >> lane) & 1) ? dz[b] : 0.0;
  const int64_t j = w * 64 + lane;
  if (j < M) part[chunk * M + j] = acc;
}

__global__ void __launch_bounds__(256) k_rhs_part(const uint64_t* __restrict__ masks, int64_t wpr, int64_t half,
                                                  int64_t M, const double* __restrict__ dz, int64_t rows_per_chunk,
                                                  double* __restrict__ part) {
  rhs_part_body(masks, wpr, half, M, dz, rows_per_chunk, part, blockIdx.x, blockIdx.y);
}

// dv[j] = sum over chunks of part[., j] (fixed order); bsum[block] = sum of its dv.
// The random rows' part of the right-hand side from their bit-transposed
// copy T (row block rb, player j: bit b = random row 64 rb + b):
// part[c][j] = sum over the kTabWords row blocks of chunk c of dzr[64 rb + b]
// over the set bits of T[rb][j], by nibble tables of dzr in LDS (entries from
// kr on are 0).  Workgroup c nxb + x; wavefront w takes player word 8 x + w,
// lane = player, so each word load is 512 contiguous bytes.
__global__ void __launch_bounds__(512) k_rhs_rand(const uint64_t* __restrict__ T, int64_t M, int64_t wpr,
                                                  int64_t kr, int64_t nrb, const double* __restrict__ dzr,
                                                  double* __restrict__ part, int64_t nxb) {
  __shared__ double tab[gnnshap::kTabWords * 256];
  const int64_t c = blockIdx.x / nxb;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t gw = (static_cast<int64_t>(blockIdx.x) % nxb) * 8 + wave;
  const int64_t b0 = c * gnnshap::kTabWords;
  const int64_t b1 = b0 + gnnshap::kTabWords < nrb ? b0 + gnnshap::kTabWords : nrb;
  const int64_t nb = b1 - b0;
  gnnshap::build_tables_bounded(dzr + b0 * 64, kr - b0 * 64, nb * 16, tab);
  __syncthreads();
  if (gw >= wpr) return;
  const int64_t j = gw * 64 + lane;
  const bool valid = j < M;
  const uint64_t* col = T + b0 * M + (valid ? j : 0);
  double acc[4] = {0.0, 0.0, 0.0, 0.0};
  gnnshap::nibble_dots<gnnshap::kTabWords>(col, M, static_cast<int>(nb), col[0], reinterpret_cast<const char*>(tab), acc);
  if (valid) part[c * M + j] = (acc[0] + acc[1]) + (acc[2] + acc[3]);
}

__global__ void __launch_bounds__(256) k_rhs_reduce(const double* __restrict__ part, int64_t nch, int64_t M,
                                                    double* __restrict__ dv, double* __restrict__ bsum) {
  __shared__ double red[256];
  const int tid = threadIdx.x;
  const int64_t j = static_cast<int64_t>(blockIdx.x) * 256 + tid;
  double v = 0.0;
  if (j < M) {
    // the chunks in order; eight loads in flight ahead of their adds
    int64_t c = 0;
    for (; c + 8 <= nch; c += 8) {
      double t[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) t[q] = part[(c + q) * M + j];
#pragma unroll
      for (int q = 0; q < 8; ++q) v += t[q];
    }
    for (; c < nch; ++c) v += part[c * M + j];
    dv[j] = v;
  }
  red[tid] = v;
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if (tid < off) red[tid] += red[tid + off];
    __syncthreads();
  }
  if (tid == 0) bsum[blockIdx.x] = red[0];
}

// rhs = P dv: subtract the mean (every block sums bsum in the same order).
__global__ void __launch_bounds__(256) k_rhs_center(const double* __restrict__ dv, const double* __restrict__ bsum,
                                                    int64_t nb, int64_t M, float* __restrict__ rhs) {
  __shared__ double mean;
  if (threadIdx.x == 0) {
    double s = 0.0;
    for (int64_t b = 0; b < nb; ++b) s += bsum[b];
    mean = s / static_cast<double>(M);
  }
  __syncthreads();
  const int64_t j = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (j < M) rhs[j] = static_cast<float>(dv[j] - mean);
}

// Right-hand side of one chunk of kTileRows representative rows, for systems
// of at most kMidMax players: part[chunk, j] = sum_b dz_b m_bj over the
// chunk, with dz_b as in dz_body.  Thread t forms dz of row chunk * kTileRows
// + t (the class found in an LDS copy of the class table) and stages the
// row's mask words; each wavefront then sums (word column, quarter of the
// chunk) items over their 64 rows in order, and the quarters are added in
// order.  Every value is fixed by the chunking alone.
__device__ __forceinline__ void rhs_tile_body(const uint64_t* __restrict__ masks, int64_t wpr, int64_t half,
                                              int64_t M, const float* __restrict__ y,
                                              const gnnshap_class* __restrict__ cls, int64_t ncls,
                                              const float* __restrict__ fef, double* __restrict__ part,
                                              int64_t chunk) {
  __shared__ int64_t c_begin[kTileClasses];
  __shared__ int32_t c_size[kTileClasses];
  __shared__ double c_weight[kTileClasses];
  __shared__ double zd[kTileRows];
  __shared__ uint32_t mw[kTileRows * 2 * kTileWords];    // row t: its 2 wpr 32-bit words
  __shared__ double qs[4 * kTileWords * 64];             // (quarter, word column, bit)
  const int t = threadIdx.x;
  const int nc = static_cast<int>(ncls), nw = static_cast<int>(2 * wpr);
  for (int i = t; i < nc; i += kTileRows) {
    c_begin[i] = cls[i].row_begin;
    c_size[i] = cls[i].size;
    c_weight[i] = cls[i].weight;
  }
  const int64_t b = chunk * kTileRows + t;
  const bool in = b < half;
  for (int w = 0; w < wpr; ++w) {
    const uint64_t word = in ? masks[b * wpr + w] : 0;
    mw[t * nw + 2 * w] = static_cast<uint32_t>(word);
    mw[t * nw + 2 * w + 1] = static_cast<uint32_t>(word >> 32);
  }
  const float yb = in ? y[b] : 0.f, yc = in ? y[b + half] : 0.f;
  __syncthreads();
  double d = 0.0;
  if (in) {
    const double Md = static_cast<double>(M);
    const double f0 = static_cast<double>(fef[0]);
    const double delta = static_cast<double>(fef[1]) - f0;
    int lo = 0, hi = nc - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (c_begin[mid] <= b) lo = mid; else hi = mid - 1;
    }
    const double w = c_weight[lo];
    const int64_t pc = c_size[lo];
    const double z1 = w * (static_cast<double>(yb) - f0 - delta / Md * static_cast<double>(pc));
    const double z2 = w * (static_cast<double>(yc) - f0 - delta / Md * static_cast<double>(M - pc));
    d = z1 - z2;
  }
  zd[t] = d;
  __syncthreads();
  const int lane = t & 63, wv = t >> 6;
  const int word = lane >> 5, bit = lane & 31;
  for (int it = wv; it < 4 * wpr; it += 4) {
    const int w = it >> 2, qq = it & 3;
    double acc = 0.0;
#pragma unroll 8
    for (int r = qq * 64; r < qq * 64 + 64; ++r) {
      const uint32_t m = mw[r * nw + 2 * w + word];
      acc = fma(static_cast<double>((m >> bit) & 1u), zd[r], acc);   // adds zd[r] exactly when the bit is set
    }
    qs[(qq * kTileWords + w) * 64 + lane] = acc;
  }
  __syncthreads();
  for (int64_t j = t; j < M; j += kTileRows) {
    const int w = static_cast<int>(j >> 6), l = static_cast<int>(j & 63);
    double sum = 0.0;
#pragma unroll
    for (int qq = 0; qq < 4; ++qq) sum += qs[(qq * kTileWords + w) * 64 + l];
    part[chunk * M + j] = sum;
  }
}

__global__ void __launch_bounds__(kTileRows) k_rhs_tile(const uint64_t* __restrict__ masks, int64_t wpr, int64_t half,
                                                        int64_t M, const float* __restrict__ y,
                                                        const gnnshap_class* __restrict__ cls, int64_t ncls,
                                                        const float* __restrict__ fef, double* __restrict__ part) {
  rhs_tile_body(masks, wpr, half, M, y, cls, ncls, fef, part, blockIdx.x);
}

// Whether a system's right-hand side takes the chunked kernel above.
bool rhs_tiled(int64_t M, int64_t ncls) { return M <= kMidMax && ncls <= kTileClasses; }

__global__ void k_zero_info(int32_t* info) { *info = 0; }

// ---- multi-block path: diagonal blocks --------------------------------------------------

constexpr int kHP = 68;                                  // LDS pitch of a 64x64 block (16-byte rows)
constexpr int kHB = 64 * kHP;                            // floats per block
constexpr size_t kPotrfLds = (5 * kHB + 64) * sizeof(float);

// One wavefront: Cholesky of a 64x64 block held row `lane` per lane in a[]
// (rows past the real block are the identity).  Column k goes through LDS
// (`col`, 64 floats): every lane reads the pivot and the entries below it as
// 16-byte broadcasts and applies the rank-1 update to its row.  Entries above
// the diagonal are left undefined.  The first non-positive pivot (1-based,
// offset o) goes to *info and is replaced by 1.
__device__ __forceinline__ void chol_wave(float (&a)[64], float* col, int64_t o, int32_t* info) {
  const int lane = threadIdx.x & 63;
  int bad = 0;
#pragma unroll
  for (int k = 0; k < 64; ++k) {
    col[lane] = a[k];
    __builtin_amdgcn_wave_barrier();
    const float piv = col[k];
    const bool ok = piv > 0.f;
    bad = (bad == 0 && !ok) ? k + 1 : bad;
    const float rs = 1.0f / sqrtf(ok ? piv : 1.f);
    a[k] *= rs;                    // L[lane][k] (lane k: sqrt of the pivot)
    const float t = a[k] * rs;     // L[lane][k] / L[k][k]: L[j][k] = col[j] rs
#pragma unroll
    for (int j4 = (k + 1) & ~3; j4 < 64; j4 += 4) {
      const f32x4 q = *reinterpret_cast<const f32x4*>(col + j4);
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (j4 + e > k) a[j4 + e] -= t * q[e];
    }
    __builtin_amdgcn_wave_barrier();
  }
  if (bad != 0 && lane == 0) atomicCAS(info, 0, static_cast<int32_t>(o + bad));
}

// One wavefront: column `lane` of W = L^-1 into w[] from Lt = L^T (pitch kHP)
// by right-looking forward substitution; row p of Lt is read as 16-byte
// broadcasts.  Entries above the diagonal come out exactly zero.
__device__ __forceinline__ void inv_wave(const float* Lt, float (&w)[64]) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int c = 0; c < 64; ++c) w[c] = c == lane ? 1.f : 0.f;
#pragma unroll
  for (int p = 0; p < 64; ++p) {
    const float* row = Lt + p * kHP;
    w[p] *= 1.0f / row[p];
    const float u = w[p];
#pragma unroll
    for (int j4 = (p + 1) & ~3; j4 < 64; j4 += 4) {
      const f32x4 q = *reinterpret_cast<const f32x4*>(row + j4);
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (j4 + e > p) w[j4 + e] -= q[e] * u;
    }
  }
}

// ---- one wavefront: Cholesky factor and its inverse of a 64x64 block -------------------
//
// Recursive 2x2 blocking on LDS blocks (pitch kHP), all in one wavefront:
//   L11 = chol(A11), W11 = L11^-1     (recursively)
//   L21 = A21 W11^T, A22 -= L21 L21^T, L22 = chol(A22), W22 = L22^-1,
//   W21 = -W22 (L21 W11),
// down to 8x8 blocks, which every lane factors and inverts in its own
// registers (no communication); the products are fp32 MFMA (32x32) or VALU.
// S <- L (zeros above the diagonal), Wb <- L^-1 (zeros above the diagonal).
// The first non-positive pivot (1-based, offset o) goes to *info and is
// replaced by 1.

__device__ __forceinline__ void chol_inv8(float* S, float* Wb, int64_t o, int32_t* info) {
  const int lane = threadIdx.x & 63;
  float a[8][8], rd[8];
#pragma unroll
  for (int r = 0; r < 8; ++r)
#pragma unroll
    for (int c = 0; c <= r; ++c) a[r][c] = S[r * kHP + c];
  int bad = 0;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    float piv = a[k][k];
#pragma unroll
    for (int q = 0; q < k; ++q) piv -= a[k][q] * a[k][q];
    const bool ok = piv > 0.f;
    bad = (bad == 0 && !ok) ? k + 1 : bad;
    const float pv = ok ? piv : 1.f;
    rd[k] = __builtin_amdgcn_rsqf(pv);     // 1/sqrt, within 1 ulp
    a[k][k] = pv * rd[k];
#pragma unroll
    for (int i = k + 1; i < 8; ++i) {
      float t = a[i][k];
#pragma unroll
      for (int q = 0; q < k; ++q) t -= a[i][q] * a[k][q];
      a[i][k] = t * rd[k];
    }
  }
  float w[8][8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    w[j][j] = rd[j];
#pragma unroll
    for (int i = j + 1; i < 8; ++i) {
      float t = 0.f;
#pragma unroll
      for (int q = j; q < i; ++q) t -= a[i][q] * w[q][j];
      w[i][j] = t * rd[i];
    }
  }
  // lane l writes element (l / 8, l % 8) of L and of W
  const int r = lane >> 3, c = lane & 7;
  float lv = 0.f, wv = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j <= i; ++j) {
      lv = (r == i && c == j) ? a[i][j] : lv;
      wv = (r == i && c == j) ? w[i][j] : wv;
    }
  __builtin_amdgcn_wave_barrier();
  S[r * kHP + c] = lv;
  Wb[r * kHP + c] = wv;
  __builtin_amdgcn_wave_barrier();
  if (bad != 0 && lane == 0 && info) atomicCAS(info, 0, static_cast<int32_t>(o + bad));
}

// One wavefront, 16 x 16 blocks: the same product as four fp32 MFMA 16x16x4.
template <bool kNT>
__device__ __forceinline__ void prod16(float* D, const float* X, const float* Y, float alpha, float beta) {
  const int lane = threadIdx.x & 63, g = lane >> 4, rl = lane & 15;
  f32x4 acc = {};
#pragma unroll
  for (int k0 = 0; k0 < 16; k0 += 4) {
    const float av = X[rl * kHP + k0 + g];
    const float bv = kNT ? Y[rl * kHP + k0 + g] : Y[(k0 + g) * kHP + rl];
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, acc, 0, 0, 0);
  }
  __builtin_amdgcn_wave_barrier();
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    float* d = D + (4 * g + r) * kHP + rl;
    *d = beta == 0.f ? alpha * acc[r] : beta * *d + alpha * acc[r];
  }
  __builtin_amdgcn_wave_barrier();
}

// One wavefront, H x H blocks (H = 8 or 16): D = alpha op(X, Y) + beta D,
// op = X Y^T (kNT) or X Y.  Every product is read before D is written, so D
// may alias X or Y.
template <int H, bool kNT>
__device__ __forceinline__ void prod_small(float* D, const float* X, const float* Y, float alpha, float beta) {
  constexpr int Q = H * H / 64;
  const int lane = threadIdx.x & 63;
  float out[Q];
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const int oi = lane + 64 * q, i = oi / H, j = oi % H;
    float sum = 0.f;
#pragma unroll
    for (int k = 0; k < H; ++k) sum += X[i * kHP + k] * (kNT ? Y[j * kHP + k] : Y[k * kHP + j]);
    out[q] = sum;
  }
  __builtin_amdgcn_wave_barrier();
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const int oi = lane + 64 * q, i = oi / H, j = oi % H;
    float* d = D + i * kHP + j;
    *d = beta == 0.f ? alpha * out[q] : beta * *d + alpha * out[q];
  }
  __builtin_amdgcn_wave_barrier();
}

// One wavefront, 32 x 32 blocks: the same product as 16 fp32 MFMA 32x32x2
// (lane half h feeds k in [16h, 16h + 16)).
template <bool kNT>
__device__ __forceinline__ void prod32(float* D, const float* X, const float* Y, float alpha, float beta) {
  const int lane = threadIdx.x & 63, h = lane >> 5, rl = lane & 31;
  f32x16 acc = {};
  const float* xr = X + rl * kHP + 16 * h;
#pragma unroll
  for (int s4 = 0; s4 < 16; s4 += 4) {
    const f32x4 a = *reinterpret_cast<const f32x4*>(xr + s4);
    f32x4 b;
    if (kNT) {
      b = *reinterpret_cast<const f32x4*>(Y + rl * kHP + 16 * h + s4);
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) b[e] = Y[(16 * h + s4 + e) * kHP + rl];
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[e], b[e], acc, 0, 0, 0);
  }
  __builtin_amdgcn_wave_barrier();
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    float* d = D + (8 * (r >> 2) + 4 * h + (r & 3)) * kHP + rl;
    *d = beta == 0.f ? alpha * acc[r] : beta * *d + alpha * acc[r];
  }
  __builtin_amdgcn_wave_barrier();
}

template <int H, bool kNT>
__device__ __forceinline__ void prod_h(float* D, const float* X, const float* Y, float alpha, float beta) {
  if constexpr (H == 32) prod32<kNT>(D, X, Y, alpha, beta);
  else if constexpr (H == 16) prod16<kNT>(D, X, Y, alpha, beta);
  else prod_small<H, kNT>(D, X, Y, alpha, beta);
}

template <int N>
__device__ __forceinline__ void chol_inv_rec(float* S, float* Wb, int64_t o, int32_t* info) {
  if constexpr (N == 8) {
    chol_inv8(S, Wb, o, info);
  } else {
    constexpr int H = N / 2;
    const int lane = threadIdx.x & 63;
    float* S21 = S + H * kHP;
    float* S22 = S21 + H;
    float* W21 = Wb + H * kHP;
    float* W22 = W21 + H;
    chol_inv_rec<H>(S, Wb, o, info);
    prod_h<H, true>(S21, S21, Wb, 1.f, 0.f);       // L21 = A21 W11^T
    prod_h<H, true>(S22, S21, S21, -1.f, 1.f);     // A22 - L21 L21^T
    chol_inv_rec<H>(S22, W22, o + H, info);
    prod_h<H, false>(W21, S21, Wb, 1.f, 0.f);      // L21 W11
    prod_h<H, false>(W21, W22, W21, -1.f, 0.f);    // W21 = -W22 (L21 W11)
    for (int t = lane; t < H * H; t += 64) {       // the upper right blocks
      S[(t / H) * kHP + H + t % H] = 0.f;
      Wb[(t / H) * kHP + H + t % H] = 0.f;
    }
    __builtin_amdgcn_wave_barrier();
  }
}

// One wavefront: S (64x64, pitch kHP) <- L = chol(S) (zeros above the
// diagonal) and Wb <- L^-1.  `col` is unused (kept for the callers' layout).
__device__ __forceinline__ void chol_inv64(float* S, float* Wb, float* col, int64_t o, int32_t* info) {
  (void)col;
  chol_inv_rec<64>(S, Wb, o, info);
}

// D = alpha op(X, Y) + beta D on 64x64 LDS blocks, op = X Y^T (kNT) or X Y;
// four wavefronts, one 32x32 quadrant each, fp32 MFMA 32x32x2 on two
// accumulator chains.  Lane half h feeds k in [32h, 32h+32), so each MFMA sums
// k and k+32.  D may alias X or Y: the products are complete before D is
// written.
template <bool kNT>
__device__ __forceinline__ void mm64(const float* X, const float* Y, float* D, float alpha, float beta) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int qr = wave >> 1, qc = wave & 1, h = lane >> 5, rl = lane & 31;
  f32x16 acc0 = {}, acc1 = {};
  const float* xr = X + (qr * 32 + rl) * kHP + h * 32;
#pragma unroll
  for (int s = 0; s < 32; s += 4) {
    const f32x4 a = *reinterpret_cast<const f32x4*>(xr + s);
    f32x4 b;
    if (kNT) {
      b = *reinterpret_cast<const f32x4*>(Y + (qc * 32 + rl) * kHP + h * 32 + s);
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) b[e] = Y[(h * 32 + s + e) * kHP + qc * 32 + rl];
    }
    acc0 = __builtin_amdgcn_mfma_f32_32x32x2f32(a[0], b[0], acc0, 0, 0, 0);
    acc1 = __builtin_amdgcn_mfma_f32_32x32x2f32(a[1], b[1], acc1, 0, 0, 0);
    acc0 = __builtin_amdgcn_mfma_f32_32x32x2f32(a[2], b[2], acc0, 0, 0, 0);
    acc1 = __builtin_amdgcn_mfma_f32_32x32x2f32(a[3], b[3], acc1, 0, 0, 0);
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    float* d = D + (qr * 32 + 8 * (r >> 2) + 4 * h + (r & 3)) * kHP + qc * 32 + rl;
    const float v = acc0[r] + acc1[r];
    *d = beta == 0.f ? alpha * v : beta * *d + alpha * v;
  }
  __syncthreads();
}

// Diagonal block at (o, o), kPB wide (identity past M), factored by 64-wide
// halves with the inverse built alongside:
//   L11 = chol(A11), W11 = L11^-1, L21 = A21 W11^T, A22 -= L21 L21^T,
//   L22 = chol(A22), W22 = L22^-1, W21 = -W22 (L21 W11).
// L goes back to the lower part of G, W = L^-1 (zero above the diagonal) to Winv.
__device__ __forceinline__ void k_potrf_body(float* G, int64_t ld, int64_t M, int64_t o, int32_t* info,
                                             float* __restrict__ Winv) {
  extern __shared__ __align__(16) unsigned char smem[];
  float* S0 = reinterpret_cast<float*>(smem);  // A11 -> L11, later L21 W11
  float* S1 = S0 + kHB;                        // W11
  float* S2 = S1 + kHB;                        // A21 -> L21, later W21
  float* S3 = S2 + kHB;                        // A22 -> L22
  float* S4 = S3 + kHB;                        // W22
  float* col = S4 + kHB;
  const int tid = threadIdx.x, wave = tid >> 6;
  const int64_t n = M - o < kPB ? M - o : kPB;
  {
    // all 64 loads of a thread in flight before the LDS stores
    float v[kPB * kPB / 256];
#pragma unroll
    for (int q = 0; q < kPB * kPB / 256; ++q) {
      const int t = tid + q * 256;
      const int r = t / kPB, c = t % kPB;
      v[q] = (r < n && c <= r) ? G[(o + r) * ld + o + c] : (r == c ? 1.f : 0.f);
    }
#pragma unroll
    for (int q = 0; q < kPB * kPB / 256; ++q) {
      const int t = tid + q * 256;
      const int r = t / kPB, c = t % kPB;
      if (r < 64 && c >= 64) continue;
      float* dst = r < 64 ? S0 + r * kHP + c : (c < 64 ? S2 + (r - 64) * kHP + c : S3 + (r - 64) * kHP + c - 64);
      *dst = v[q];
    }
  }
  __syncthreads();
  if (wave == 0) chol_inv64(S0, S1, col, o, info);
  __syncthreads();
  mm64<true>(S2, S1, S2, 1.f, 0.f);     // L21
  mm64<true>(S2, S2, S3, -1.f, 1.f);    // A22 - L21 L21^T
  for (int t = tid; t < kPB * 64; t += 256) {
    const int r = t / 64, c = t % 64;
    if (r < n && c < n && c <= r) G[(o + r) * ld + o + c] = r < 64 ? S0[r * kHP + c] : S2[(r - 64) * kHP + c];
  }
  __syncthreads();
  mm64<false>(S2, S1, S0, 1.f, 0.f);    // L21 W11
  if (wave == 0) chol_inv64(S3, S4, col, o + 64, info);
  __syncthreads();
  mm64<false>(S4, S0, S2, -1.f, 0.f);   // W21
  for (int t = tid; t < 64 * 64; t += 256) {
    const int r = t / 64, c = t % 64;
    if (64 + r < n && 64 + c < n && c <= r) G[(o + 64 + r) * ld + o + 64 + c] = S3[r * kHP + c];
  }
  for (int t = tid; t < kPB * kPB; t += 256) {
    const int r = t / kPB, c = t % kPB;
    float v;
    if (r < 64) v = c < 64 ? S1[r * kHP + c] : 0.f;
    else v = c < 64 ? S2[(r - 64) * kHP + c] : S4[(r - 64) * kHP + c - 64];
    Winv[t] = v;
  }
}

__global__ void __launch_bounds__(256) k_potrf(float* G, int64_t ld, int64_t M, int64_t o, int32_t* info,
                                               float* __restrict__ Winv) {
  k_potrf_body(G, ld, M, o, info, Winv);
}

// ---- one-workgroup path (systems of up to kMidMax players) --------------------------------
//
// G~ is assembled in global memory by multi-block kernels (L2-resident at
// these sizes) and one workgroup of four wavefronts factors it in 64-wide
// panels.  Per panel:
// the panel blocks are loaded at once; L_Ip = A_Ip W_pp^T as MFMA products
// (W_pp = L_pp^-1, one task per 32-row half); the forward substitution rides
// along (z_p = W_pp r_p, r_I -= L_Ip z_p); the trailing tiles of the next
// panel's block column are updated first, then wavefront 0 factors and
// inverts the next diagonal block (wavefront Cholesky with LDS column
// broadcasts) while the other three update the rest of the trailing matrix
// in 32x32 MFMA tiles.  The backward substitution reads L and the stored
// inverses once more.

constexpr int kMidThreads = 256;
constexpr int kMidBlk = kMidMax / 64;
constexpr size_t kMidLds = (static_cast<size_t>(1 + kMidBlk) * kHB + 64 + kMidMax + 4 * 64) * sizeof(float);

// G: G~ on its lower triangle (row stride ld) on entry, the factor on exit;
// dvg: the summed right-hand side before centring; Wd: room for the
// ceil(M/64) inverse diagonal factors.
__device__ __forceinline__ void solve_mid_body(float* G, int64_t ld, int64_t M, const double* __restrict__ dvg,
                                               const float* __restrict__ fef, float* __restrict__ Wd, int32_t* info,
                                               float* __restrict__ phi) {
  constexpr int NT = kMidThreads, NW = NT / 64;
  extern __shared__ __align__(16) unsigned char smem[];
  float* D0 = reinterpret_cast<float*>(smem);  // diagonal block -> L_pp (and the look-ahead's)
  float* D1 = D0 + kHB;                        // W_pp = L_pp^-1
  float* P = D1 + kHB;                         // blocks below the diagonal block -> L_Ip
  float* col = P + (kMidBlk - 1) * kHB;        // 64: column broadcasts of the wavefront Cholesky
  float* rv = col + 64;                        // kMidMax: r, then z, then psi
  float* red8 = rv + kMidMax;                  // NW x 64
  __shared__ double red[NW];
  __shared__ double sc[2];                     // mean of dv, Delta
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int h = lane >> 5, rl = lane & 31;
  const double Md = static_cast<double>(M);
  const int64_t nblk = (M + 63) / 64;
  if (tid == 0) *info = 0;

  // 1. the centred right-hand side r = P dv
  double sv = 0.0;
  for (int64_t i = tid; i < M; i += NT) sv += dvg[i];
  for (int off = 32; off > 0; off >>= 1) sv += __shfl_xor(sv, off);
  if (lane == 0) red[wave] = sv;
  __syncthreads();
  if (tid == 0) {
    double t = 0.0;
    for (int w = 0; w < NW; ++w) t += red[w];
    sc[0] = t / Md;
    sc[1] = static_cast<double>(fef[1]) - static_cast<double>(fef[0]);
  }
  __syncthreads();
  for (int64_t i = tid; i < nblk * 64; i += NT) rv[i] = i < M ? static_cast<float>(dvg[i] - sc[0]) : 0.f;
  const int ldi = static_cast<int>(ld);       // M <= kMidMax: 32-bit offsets within G
  // one wavefront: the 64x64 diagonal block at (o, o) into D0 (lower part,
  // identity past M), then D0 <- L, D1 <- L^-1
  auto diag_factor = [&](int64_t o) {
    const float* base = G + o * ld + o;
#pragma unroll
    for (int h2 = 0; h2 < 64; h2 += 32) {
      float v[32];
#pragma unroll
      for (int q = 0; q < 32; ++q) {
        const int r = h2 + q;
        const bool ok = o + r < M && lane <= r;
        v[q] = ok ? base[r * ldi + lane] : 0.f;
      }
#pragma unroll
      for (int q = 0; q < 32; ++q) {
        const int r = h2 + q;
        float x = v[q];
        if (o + r >= M && r == lane) x = 1.f;
        D0[r * kHP + lane] = x;
      }
    }
    __builtin_amdgcn_wave_barrier();
    chol_inv64(D0, D1, col, o, info);
  };
  // one task: trailing quadrant (qr, qc) of tile (I, J) below panel o: A -= L_Io L_Jo^T
  auto trailing = [&](int64_t o, int I, int J, int q) {
    const int qr = q >> 1, qc = q & 1;
    if (I == J && qr < qc) return;
    const int64_t gi0 = o + 64 * (I + 1) + 32 * qr, gj = o + 64 * (J + 1) + 32 * qc + rl;
    float* tile = G + gi0 * ld + (gj - rl);
    f32x16 acc;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int rr = 8 * (r >> 2) + 4 * h + (r & 3);
      const bool ok = gi0 + rr < M && gj < M;
      acc[r] = ok ? tile[rr * ldi + rl] : 0.f;
    }
    const float* xa = P + I * kHB + (32 * qr + rl) * kHP + h * 32;
    const float* xb = P + J * kHB + (32 * qc + rl) * kHP + h * 32;
#pragma unroll
    for (int s4 = 0; s4 < 32; s4 += 4) {
      const f32x4 a = *reinterpret_cast<const f32x4*>(xa + s4);
      const f32x4 b = *reinterpret_cast<const f32x4*>(xb + s4);
#pragma unroll
      for (int e = 0; e < 4; ++e) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(-a[e], b[e], acc, 0, 0, 0);
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int rr = 8 * (r >> 2) + 4 * h + (r & 3);
      if (gi0 + rr < M && gj < M) tile[rr * ldi + rl] = acc[r];
    }
  };
  __syncthreads();

  // 2. factorisation with the forward substitution; "panel -1" only factors
  // the first diagonal block
  for (int64_t p = -1; p < nblk; ++p) {
    const int64_t o = p * 64;
    const int nI = static_cast<int>(nblk - p - 1);
    if (p >= 0) {
    // (a) the blocks below the diagonal block, three blocks' loads in flight at a time
    {
      constexpr int QB = 4096 / NT;
      const float* base = G + (o + 64) * ld + o;
      for (int I0 = 0; I0 < nI; I0 += 3) {
        float v[3][QB];
#pragma unroll
        for (int ii = 0; ii < 3; ++ii)
#pragma unroll
          for (int q = 0; q < QB; ++q) {
            const int t = tid + q * NT;
            const int r = 64 * (I0 + ii) + (t >> 6);
            v[ii][q] = (I0 + ii < nI && o + 64 + r < M) ? base[r * ldi + (t & 63)] : 0.f;
          }
#pragma unroll
        for (int ii = 0; ii < 3; ++ii) {
          if (I0 + ii >= nI) break;
#pragma unroll
          for (int q = 0; q < QB; ++q) {
            const int t = tid + q * NT;
            P[(I0 + ii) * kHB + (t >> 6) * kHP + (t & 63)] = v[ii][q];
          }
        }
      }
    }
    // (b) z_p = W_pp r_p; L_pp and W_pp to global
    if (wave == 0) {
      float z = 0.f;
#pragma unroll 8
      for (int c = 0; c < 64; ++c) z += D1[lane * kHP + c] * rv[o + c];
      __builtin_amdgcn_wave_barrier();
      rv[o + lane] = z;
    }
    for (int t = tid; t < 64 * 64; t += NT) {
      const int r = t >> 6, c = t & 63;
      const int64_t gi = o + r, gj = o + c;
      if (gi < M && gj <= gi) G[gi * ld + gj] = D0[r * kHP + c];
      Wd[p * 4096 + t] = D1[r * kHP + c];
    }
    __syncthreads();
    // (c) L_Ip = A_Ip W_pp^T, one task per 32-row half of a block
    for (int task = wave; task < 2 * nI; task += NW) {
      const int I = task >> 1, qr = task & 1;
      float* blk = P + I * kHB;
      f32x16 a0 = {}, a1 = {};
      const float* xr = blk + (32 * qr + rl) * kHP + h * 32;
#pragma unroll
      for (int s4 = 0; s4 < 32; s4 += 4) {
        const f32x4 a = *reinterpret_cast<const f32x4*>(xr + s4);
        const f32x4 b0 = *reinterpret_cast<const f32x4*>(D1 + rl * kHP + h * 32 + s4);
        const f32x4 b1 = *reinterpret_cast<const f32x4*>(D1 + (32 + rl) * kHP + h * 32 + s4);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          a0 = __builtin_amdgcn_mfma_f32_32x32x2f32(a[e], b0[e], a0, 0, 0, 0);
          a1 = __builtin_amdgcn_mfma_f32_32x32x2f32(a[e], b1[e], a1, 0, 0, 0);
        }
      }
      __builtin_amdgcn_wave_barrier();
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float* d = blk + (32 * qr + 8 * (r >> 2) + 4 * h + (r & 3)) * kHP + rl;
        d[0] = a0[r];
        d[32] = a1[r];
      }
    }
    __syncthreads();
    // (d) r_I -= L_Ip z_p; L_Ip to global
    for (int R = tid; R < nI * 64; R += NT) {
      const float* pr = P + (R >> 6) * kHB + (R & 63) * kHP;
      float sum = 0.f;
#pragma unroll 8
      for (int c = 0; c < 64; ++c) sum += pr[c] * rv[o + c];
      rv[o + 64 + R] -= sum;
    }
    for (int I = 0; I < nI; ++I)
      for (int t = tid; t < 64 * 64; t += NT) {
        const int r = t >> 6, c = t & 63;
        const int64_t gi = o + 64 * (I + 1) + r;
        if (gi < M) G[gi * ld + o + c] = P[I * kHB + r * kHP + c];
      }
    // (e) the next panel's block column first
    for (int task = wave; task < 4 * nI; task += NW) trailing(o, task >> 2, 0, task & 3);
    __syncthreads();
    }
    // (f) wavefront 0 factors the next diagonal block; the others update the rest
    if (nI > 0) {
      if (wave == 0) {
        diag_factor(o + 64);
      } else if (p >= 0) {
        const int tasks = 4 * (nI * (nI - 1) / 2);
        for (int task = wave - 1; task < tasks; task += NW - 1) {
          const int pair = task >> 2;
          int I1 = 0;
          while ((I1 + 1) * (I1 + 2) / 2 <= pair) ++I1;
          const int J1 = pair - I1 * (I1 + 1) / 2;
          trailing(o, I1 + 1, J1 + 1, task & 3);
        }
      }
    }
    __syncthreads();
  }

  // 3. backward substitution: psi_p = W_pp^T (z_p - sum_I L_Ip^T psi_I)
  for (int64_t p = nblk - 1; p >= 0; --p) {
    const int64_t o = p * 64;
    const int c = tid & 63, g = tid >> 6;
    const bool real = o + c < M;      // columns past M (row padding of G) are never read
    float acc = 0.f;
    if (real) {
#pragma unroll 8
      for (int64_t row = o + 64 + g; row < M; row += NW) acc += G[row * ld + o + c] * rv[row];
    }
    red8[g * 64 + c] = acc;
    __syncthreads();
    if (tid < 64) {
      float sum = 0.f;
      for (int gg = 0; gg < NW; ++gg) sum += red8[gg * 64 + tid];
      red8[tid] = o + tid < M ? rv[o + tid] - sum : 0.f;
    }
    __syncthreads();
    if (tid < 64) {
      float ps = 0.f;
#pragma unroll 8
      for (int cc = tid; cc < 64; ++cc) ps += Wd[p * 4096 + cc * 64 + tid] * red8[cc];
      rv[o + tid] = ps;
    }
    __syncthreads();
  }
  const double delta = sc[1];
  for (int64_t i = tid; i < M; i += NT) phi[i] = static_cast<float>(delta / Md + static_cast<double>(rv[i]));
}

__global__ void __launch_bounds__(kMidThreads) k_solve_mid(float* G, int64_t ld, int64_t M,
                                                           const double* __restrict__ dvg,
                                                           const float* __restrict__ fef, float* __restrict__ Wd,
                                                           int32_t* info, float* __restrict__ phi) {
  solve_mid_body(G, ld, M, dvg, fef, Wd, info, phi);
}

// ---- multi-block path: MFMA GEMM ---------------------------------------------------------

constexpr int kGT = 128;        // output tile edge
constexpr int kGK = 32;         // K chunk staged in LDS
constexpr int kGP = kGK + 4;    // LDS row pitch (floats)

// C = beta C + alpha A B^T over 128x128 tiles, fp32 MFMA 32x32x2; rows of A and
// B are K contiguous floats (K a multiple of 32; lda, ldb multiples of 4 and
// 16-byte aligned bases).  Four wavefronts own 64x64 quadrants; lane half h
// feeds k in [16h, 16h+16) of each chunk.  kLower: blockIdx.x enumerates the
// tiles with J <= I (diagonal tiles written whole).  A may alias C when one
// tile column covers all of n (the tile reads its rows before writing them).
template <bool kLower>
__device__ __forceinline__ void k_gemm_nt_body(const float* A, int64_t lda, const float* B, int64_t ldb, float* C,
                                               int64_t ldc, int64_t m, int64_t n, int64_t K, float alpha,
                                               float beta, int64_t tiles_n, int64_t bx) {
  __shared__ __align__(16) float As[kGT * kGP];
  __shared__ __align__(16) float Bs[kGT * kGP];
  const int64_t t = bx;
  int64_t I, J;
  if (kLower) {
    I = static_cast<int64_t>((sqrt(8.0 * static_cast<double>(t) + 1.0) - 1.0) * 0.5);
    while (I * (I + 1) / 2 > t) --I;
    while ((I + 1) * (I + 2) / 2 <= t) ++I;
    J = t - I * (I + 1) / 2;
  } else {
    I = t / tiles_n;
    J = t % tiles_n;
  }
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = wave >> 1, wc = wave & 1, h = lane >> 5, rl = lane & 31;
  const int64_t i0 = I * kGT, j0 = J * kGT;
  f32x16 acc[2][2];
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y) acc[x][y] = f32x16{};
  for (int64_t p0 = 0; p0 < K; p0 += kGK) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int idx = tid + q * 256;
      const int r = idx >> 3, c4 = (idx & 7) << 2;
      f32x4 va = {0.f, 0.f, 0.f, 0.f}, vb = {0.f, 0.f, 0.f, 0.f};
      if (i0 + r < m) va = *reinterpret_cast<const f32x4*>(A + (i0 + r) * lda + p0 + c4);
      if (j0 + r < n) vb = *reinterpret_cast<const f32x4*>(B + (j0 + r) * ldb + p0 + c4);
      *reinterpret_cast<f32x4*>(As + r * kGP + c4) = va;
      *reinterpret_cast<f32x4*>(Bs + r * kGP + c4) = vb;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; kk += 4) {
      f32x4 a[2], b[2];
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        a[s] = *reinterpret_cast<const f32x4*>(As + (wr * 64 + s * 32 + rl) * kGP + h * 16 + kk);
        b[s] = *reinterpret_cast<const f32x4*>(Bs + (wc * 64 + s * 32 + rl) * kGP + h * 16 + kk);
      }
#pragma unroll
      for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int x = 0; x < 2; ++x)
#pragma unroll
          for (int y = 0; y < 2; ++y)
            acc[x][y] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[x][e], b[y][e], acc[x][y], 0, 0, 0);
    }
    __syncthreads();
  }
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y) {
      const int64_t col = j0 + wc * 64 + y * 32 + rl;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = i0 + wr * 64 + x * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
        if (row < m && col < n) {
          float* c = C + row * ldc + col;
          *c = beta == 0.f ? alpha * acc[x][y][r] : beta * *c + alpha * acc[x][y][r];
        }
      }
    }
}

template <bool kLower>
__global__ void __launch_bounds__(256) k_gemm_nt(const float* A, int64_t lda, const float* B, int64_t ldb, float* C,
                                                 int64_t ldc, int64_t m, int64_t n, int64_t K, float alpha,
                                                 float beta, int64_t tiles_n) {
  k_gemm_nt_body<kLower>(A, lda, B, ldb, C, ldc, m, n, K, alpha, beta, tiles_n, blockIdx.x);
}

// ---- multi-block path: triangular solves ------------------------------------------------
//
// Segments [s0, s1) of at most kSeg rows: one workgroup loads the segment's
// lower triangle into LDS (packed, row i at i(i+1)/2) and substitutes through
// it in 64-row blocks (one wavefront per diagonal block); multi-block GEMVs
// then carry the segment's unknowns to the rows outside it.

__device__ __forceinline__ int64_t tri(int64_t i, int64_t j) { return ((i * (i + 1)) >> 1) + j; }

constexpr size_t kTrsvLds = (kSeg * (kSeg + 1) / 2 + 2 * kSeg) * sizeof(float);

// Packed triangle of rows/cols [s0, s1) and reciprocal pivots, all loads in flight at once.
__device__ __forceinline__ void load_segment(const float* __restrict__ G, int64_t ld, int64_t s0, int64_t len, float* Ls,
                                    float* rd) {
  const int64_t total = len * (len + 1) / 2;
  constexpr int kPer = (kSeg * (kSeg + 1) / 2 + 1023) / 1024;
  float v[kPer];
#pragma unroll
  for (int q = 0; q < kPer; ++q) {
    const int64_t t = threadIdx.x + static_cast<int64_t>(q) * 1024;
    int64_t i = static_cast<int64_t>((sqrtf(8.f * static_cast<float>(t) + 1.f) - 1.f) * 0.5f);
    if (i * (i + 1) / 2 > t) --i;
    if ((i + 1) * (i + 2) / 2 <= t) ++i;
    const int64_t j = t - i * (i + 1) / 2;
    v[q] = t < total ? G[(s0 + i) * ld + s0 + j] : 0.f;
  }
#pragma unroll
  for (int q = 0; q < kPer; ++q) {
    const int64_t t = threadIdx.x + static_cast<int64_t>(q) * 1024;
    if (t < total) Ls[t] = v[q];
  }
  __syncthreads();
  for (int64_t i = threadIdx.x; i < len; i += blockDim.x) rd[i] = 1.0f / Ls[tri(i, i)];
  __syncthreads();
}

// Forward: x[s0:s1) = L[s0:s1, s0:s1)^-1 rhs[s0:s1) (rhs holds the earlier segments' updates).
__device__ __forceinline__ void k_trsv_fwd_body(const float* __restrict__ G, int64_t ld, int64_t s0, int64_t s1,
                                                const float* __restrict__ rhs, float* __restrict__ x) {
  extern __shared__ __align__(16) unsigned char smem[];
  float* Ls = reinterpret_cast<float*>(smem);
  float* rd = Ls + kSeg * (kSeg + 1) / 2;
  float* v = rd + kSeg;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, nw = blockDim.x >> 6;
  const int64_t len = s1 - s0;
  for (int64_t t = tid; t < len; t += blockDim.x) v[t] = rhs[s0 + t];
  load_segment(G, ld, s0, len, Ls, rd);
  for (int64_t ob = 0; ob < len; ob += kTB) {
    const int nbe = static_cast<int>(len - ob < kTB ? len - ob : kTB);
    if (wave == 0) {
      // b_k is final once the columns before k are applied: x_k = b_k / L_kk
      const int r = lane < nbe ? lane : 0;
      float b = lane < nbe ? v[ob + lane] : 0.f;
      float lr[kTB];
#pragma unroll
      for (int c = 0; c < kTB; ++c) lr[c] = (lane < nbe && c < lane) ? Ls[tri(ob + r, ob + c)] : 0.f;
#pragma unroll
      for (int k = 0; k < kTB; ++k) {
        const float rk = k < nbe ? rd[ob + k] : 1.f;
        b -= lr[k] * (bcast(b, k) * rk);
      }
      if (lane < nbe) v[ob + lane] = b * rd[ob + lane];
    }
    __syncthreads();
    const float xo = lane < nbe ? v[ob + lane] : 0.f;
    for (int64_t i = ob + nbe + wave; i < len; i += nw) {
      const float p = wave_sum(lane < nbe ? Ls[tri(i, ob) + lane] * xo : 0.f);
      if (lane == 0) v[i] -= p;
    }
    __syncthreads();
  }
  for (int64_t t = tid; t < len; t += blockDim.x) x[s0 + t] = v[t];
}

__global__ void __launch_bounds__(1024) k_trsv_fwd(const float* __restrict__ G, int64_t ld, int64_t s0, int64_t s1,
                                                   const float* __restrict__ rhs, float* __restrict__ x) {
  k_trsv_fwd_body(G, ld, s0, s1, rhs, x);
}

// rhs[i] -= L[i, s0:s1) x[s0:s1) for i >= s1; one wavefront per row, four floats per lane.
__device__ __forceinline__ void k_gemv_fwd_body(const float* __restrict__ G, int64_t ld, int64_t M, int64_t s0,
                                                int64_t s1, const float* __restrict__ x, float* __restrict__ rhs, int64_t bx) {
  const int lane = threadIdx.x & 63;
  const int64_t i = s1 + ((static_cast<int64_t>(bx) * blockDim.x + threadIdx.x) >> 6);
  if (i >= M) return;
  float acc = 0.f;
  for (int64_t c = s0 + 4 * lane; c < s1; c += 256) {
    if (c + 4 <= s1) {
      const f32x4 g = *reinterpret_cast<const f32x4*>(G + i * ld + c);
      const f32x4 xv = *reinterpret_cast<const f32x4*>(x + c);
      acc += g[0] * xv[0] + g[1] * xv[1] + g[2] * xv[2] + g[3] * xv[3];
    } else {
      for (int64_t e = c; e < s1; ++e) acc += G[i * ld + e] * x[e];
    }
  }
  acc = wave_sum(acc);
  if (lane == 0) rhs[i] -= acc;
}

__global__ void __launch_bounds__(256) k_gemv_fwd(const float* __restrict__ G, int64_t ld, int64_t M, int64_t s0,
                                                  int64_t s1, const float* __restrict__ x, float* __restrict__ rhs) {
  k_gemv_fwd_body(G, ld, M, s0, s1, x, rhs, blockIdx.x);
}

// Backward: z[s0:s1) = L[s0:s1, s0:s1)^-T x[s0:s1) into rhs (x holds the later segments' updates).
__device__ __forceinline__ void k_trsv_bwd_body(const float* __restrict__ G, int64_t ld, int64_t s0, int64_t s1,
                                                const float* __restrict__ x, float* __restrict__ rhs) {
  extern __shared__ __align__(16) unsigned char smem[];
  float* Ls = reinterpret_cast<float*>(smem);
  float* rd = Ls + kSeg * (kSeg + 1) / 2;
  float* v = rd + kSeg;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int64_t len = s1 - s0;
  for (int64_t t = tid; t < len; t += blockDim.x) v[t] = x[s0 + t];
  load_segment(G, ld, s0, len, Ls, rd);
  for (int64_t ob = ((len - 1) / kTB) * kTB; ob >= 0; ob -= kTB) {
    const int nbe = static_cast<int>(len - ob < kTB ? len - ob : kTB);
    if (wave == 0) {
      // lc[k] = L[ob+k][ob+lane] for k > lane: column `lane` of the block
      const int r = lane < nbe ? lane : 0;
      float b = lane < nbe ? v[ob + lane] : 0.f;
      float lc[kTB];
#pragma unroll
      for (int k = 0; k < kTB; ++k) lc[k] = (lane < nbe && k > lane && k < nbe) ? Ls[tri(ob + k, ob + r)] : 0.f;
#pragma unroll
      for (int k = kTB - 1; k >= 0; --k) {
        const float rk = k < nbe ? rd[ob + k] : 1.f;
        b -= lc[k] * (bcast(b, k) * rk);
      }
      if (lane < nbe) v[ob + lane] = b * rd[ob + lane];
    }
    __syncthreads();
    for (int64_t i = tid; i < ob; i += blockDim.x) {
      float acc = 0.f;
      for (int c = 0; c < nbe; ++c) acc += Ls[tri(ob + c, i)] * v[ob + c];
      v[i] -= acc;
    }
    __syncthreads();
  }
  for (int64_t t = tid; t < len; t += blockDim.x) rhs[s0 + t] = v[t];
}

__global__ void __launch_bounds__(1024) k_trsv_bwd(const float* __restrict__ G, int64_t ld, int64_t s0, int64_t s1,
                                                   const float* __restrict__ x, float* __restrict__ rhs) {
  k_trsv_bwd_body(G, ld, s0, s1, x, rhs);
}

// x[i] -= sum_{c in [s0, s1)} L[c, i] z[c] for i < s0: 64 rows i per block
// (coalesced over i), the segment split over four thread groups.
__device__ __forceinline__ void k_gemv_bwd_body(const float* __restrict__ G, int64_t ld, int64_t s0, int64_t s1,
                                                const float* __restrict__ z, float* __restrict__ x, int64_t bx) {
  __shared__ float red[4][64];
  const int il = threadIdx.x & 63, g = threadIdx.x >> 6;
  const int64_t i = static_cast<int64_t>(bx) * 64 + il;
  float acc = 0.f;
  if (i < s0) {
#pragma unroll 8
    for (int64_t c = s0 + g; c < s1; c += 4) acc += G[c * ld + i] * z[c];
  }
  red[g][il] = acc;
  __syncthreads();
  if (g == 0 && i < s0) x[i] -= (red[0][il] + red[1][il]) + (red[2][il] + red[3][il]);
}

__global__ void __launch_bounds__(256) k_gemv_bwd(const float* __restrict__ G, int64_t ld, int64_t s0, int64_t s1,
                                                  const float* __restrict__ z, float* __restrict__ x) {
  k_gemv_bwd_body(G, ld, s0, s1, z, x, blockIdx.x);
}

__device__ __forceinline__ void k_finish_body(const float* __restrict__ z, int64_t M, const double* __restrict__ scal,
                                              float* __restrict__ phi, int64_t bx, int64_t gx) {
  const double base = scal[3] / static_cast<double>(M);
  for (int64_t i = static_cast<int64_t>(bx) * blockDim.x + threadIdx.x; i < M;
       i += static_cast<int64_t>(gx) * blockDim.x)
    phi[i] = static_cast<float>(base + static_cast<double>(z[i]));
}

__global__ void k_finish(const float* __restrict__ z, int64_t M, const double* __restrict__ scal,
                         float* __restrict__ phi) {
  k_finish_body(z, M, scal, phi, blockIdx.x, gridDim.x);
}

// ---- multi-block path, batched: one system per blockIdx.y ---------------------------------
//
// Every launch covers the step of the largest system; a system whose M ends
// before the step returns at once (whole workgroups, before any barrier), so
// each system sees exactly the launches, grids and arguments it would see
// alone and its factor and phi are the same bits.

__global__ void __launch_bounds__(256) k_potrf_mb(const gnnshap::MbJob* __restrict__ jobs, int64_t o) {
  const gnnshap::MbJob J = jobs[blockIdx.y];
  if (o >= J.M) return;
  k_potrf_body(J.G, J.ld, J.M, o, J.info, J.Winv);
}

// panel <- panel W^T (the off-diagonal blocks of the step's 128 columns)
__global__ void __launch_bounds__(256) k_trsm_mb(const gnnshap::MbJob* __restrict__ jobs, int64_t o) {
  const gnnshap::MbJob J = jobs[blockIdx.y];
  const int64_t r0 = o + kPB;
  if (r0 >= J.M) return;
  const int64_t rows = J.M - r0;
  if (static_cast<int64_t>(blockIdx.x) >= (rows + kGT - 1) / kGT) return;
  float* panel = J.G + r0 * J.ld + o;
  k_gemm_nt_body<false>(panel, J.ld, J.Winv, kPB, panel, J.ld, rows, kPB, kPB, 1.f, 0.f, 1, blockIdx.x);
}

// trailing lower triangle -= panel panel^T
__global__ void __launch_bounds__(256) k_syrk_mb(const gnnshap::MbJob* __restrict__ jobs, int64_t o) {
  const gnnshap::MbJob J = jobs[blockIdx.y];
  const int64_t r0 = o + kPB;
  if (r0 >= J.M) return;
  const int64_t rows = J.M - r0;
  const int64_t tr = (rows + kGT - 1) / kGT;
  if (static_cast<int64_t>(blockIdx.x) >= tr * (tr + 1) / 2) return;
  const float* panel = J.G + r0 * J.ld + o;
  k_gemm_nt_body<true>(panel, J.ld, panel, J.ld, J.G + r0 * J.ld + r0, J.ld, rows, rows, kPB, -1.f, 1.f, 0,
                       blockIdx.x);
}

__global__ void __launch_bounds__(1024) k_trsv_fwd_mb(const gnnshap::MbJob* __restrict__ jobs, int64_t s0) {
  const gnnshap::MbJob J = jobs[blockIdx.y];
  if (s0 >= J.M) return;
  k_trsv_fwd_body(J.G, J.ld, s0, J.M < s0 + kSeg ? J.M : s0 + kSeg, J.rhs, J.x);
}

__global__ void __launch_bounds__(256) k_gemv_fwd_mb(const gnnshap::MbJob* __restrict__ jobs, int64_t s0) {
  const gnnshap::MbJob J = jobs[blockIdx.y];
  const int64_t s1 = s0 + kSeg;
  if (s1 >= J.M) return;
  k_gemv_fwd_body(J.G, J.ld, J.M, s0, s1, J.x, J.rhs, blockIdx.x);
}

__global__ void __launch_bounds__(1024) k_trsv_bwd_mb(const gnnshap::MbJob* __restrict__ jobs, int64_t s0) {
  const gnnshap::MbJob J = jobs[blockIdx.y];
  if (s0 >= J.M) return;
  k_trsv_bwd_body(J.G, J.ld, s0, J.M < s0 + kSeg ? J.M : s0 + kSeg, J.x, J.rhs);
}

__global__ void __launch_bounds__(256) k_gemv_bwd_mb(const gnnshap::MbJob* __restrict__ jobs, int64_t s0) {
  const gnnshap::MbJob J = jobs[blockIdx.y];
  if (s0 >= J.M) return;
  k_gemv_bwd_body(J.G, J.ld, s0, J.M < s0 + kSeg ? J.M : s0 + kSeg, J.rhs, J.x, blockIdx.x);
}

__global__ void k_finish_mb(const gnnshap::MbJob* __restrict__ jobs) {
  const gnnshap::MbJob J = jobs[blockIdx.y];
  k_finish_body(J.rhs, J.M, J.scal, J.phi, blockIdx.x, gridDim.x);
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

// ---- multi-target path (one-workgroup systems): one job per blockIdx.y / .z --------------

// Also clears the count matrix (M rows of ld) for the Gram's atomics: the
// job's nrb x wpr workgroups each clear an equal share of it.
// Jobs of at most kGramWhole random row words get each count from one
// workgroup (plain stores); larger ones are split over chunks of kGramChunk
// words whose partial counts are added with integer atomics into zeroed counts.
constexpr int64_t kGramChunk = 32;
constexpr int64_t kGramWhole = 128;

// One wavefront per transpose item of the batch (four per workgroup): item g
// belongs to the job with the largest tr0 <= g (a wavefront-wide search of
// the job table), as (row block, word) = divmod(g - tr0, wpr).
constexpr int kTrWaves = 4;
__global__ void __launch_bounds__(kTrWaves * 64) k_transpose_batch(const gnnshap::SolveJob* __restrict__ jobs,
                                                                   int64_t n, int64_t n_items) {
  const int lane = threadIdx.x & 63;
  const int64_t g = static_cast<int64_t>(blockIdx.x) * kTrWaves + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (g >= n_items) return;
  int64_t lo = 0, hi = n;   // jobs[lo].tr0 <= g < jobs[hi].tr0 (jobs[n].tr0 = infinity)
  while (hi - lo > 1) {
    const int64_t step = (hi - lo + 63) / 64;
    const int64_t idx = lo + lane * step;
    const bool ok = idx < hi && jobs[idx].tr0 <= g;
    const uint64_t m = __ballot(ok);
    const int64_t last = 63 - __clzll(static_cast<long long>(m));
    lo += last * step;
    hi = lo + step < hi ? lo + step : hi;
  }
  const gnnshap::SolveJob& J = jobs[lo];
  const int64_t item = g - J.tr0;
  const int64_t rb = item / J.wpr, w = item % J.wpr;
  transpose_body(J.masks, J.wpr, J.rb0, J.kr, J.M, J.T, rb, w);
  if (item == 0)       // the Gram adds its row sums into usum
    for (int64_t i = lane; i < J.M; i += 64) J.usum[i] = 0;
  if (J.nrb <= kGramWhole) return;             // every count is stored by one workgroup
  const int64_t nblk = J.nrb * J.wpr;
  const int64_t total = J.M * J.ld, per = (total + nblk - 1) / nblk;
  const int64_t e0 = item * per, e1 = e0 + per < total ? e0 + per : total;
  for (int64_t e = e0 + lane; e < e1; e += 64) J.counts[e] = 0;
}

// Workgroup (tile, chunk, job): tile = J' (J' + 1) / 2 + I' over the tiles
// I' <= J' of the job, chunk = kGramChunk row words (chunk 0 only when the
// job's counts are whole).
__global__ void __launch_bounds__(256) k_gram_batch(const gnnshap::SolveJob* __restrict__ jobs) {
  const gnnshap::SolveJob J = jobs[blockIdx.z];
  const int64_t nb = (J.M + 63) / 64;
  const int64_t tile = blockIdx.x, w0 = static_cast<int64_t>(blockIdx.y) * kGramChunk;
  const bool whole = J.nrb <= kGramWhole;
  if (J.kr <= 0 || tile >= nb * (nb + 1) / 2 || w0 >= J.nrb || (whole && blockIdx.y > 0)) return;
  int64_t Jt = 0;
  while ((Jt + 1) * (Jt + 2) / 2 <= tile) ++Jt;
  const int64_t It = tile - Jt * (Jt + 1) / 2;
  if (whole)
    gram_body(J.T, J.nrb, J.M, J.ld, J.counts, It, Jt, J.usum);
  else
    gram_part_body(J.T, w0, w0 + kGramChunk < J.nrb ? w0 + kGramChunk : J.nrb, J.M, J.ld, J.counts, It, Jt, J.usum);
}

__global__ void __launch_bounds__(kTileRows) k_rhs_tile_batch(const gnnshap::SolveJob* __restrict__ jobs) {
  const gnnshap::SolveJob J = jobs[blockIdx.y];
  if (blockIdx.x >= J.nch) return;
  rhs_tile_body(J.masks, J.wpr, J.half, J.M, J.y, J.cls, J.ncls, J.fef, J.part, blockIdx.x);
}

__global__ void __launch_bounds__(256) k_rhs_sum_batch(const gnnshap::SolveJob* __restrict__ jobs) {
  const gnnshap::SolveJob J = jobs[blockIdx.y];
  const int64_t j = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (j >= J.M) return;
  double v = 0.0;
  for (int64_t c = 0; c < J.nch; ++c) v += J.part[c * J.M + j];
  J.dv[j] = v;
}

__global__ void __launch_bounds__(256) k_scalars_batch(const gnnshap::SolveJob* __restrict__ jobs) {
  const gnnshap::SolveJob J = jobs[blockIdx.x];
  scalars_body(J.counts, J.usum, J.M, J.ld, J.kr > 0, J.alpha, J.wr, nullptr, J.scal);   // G~ only
}

__global__ void __launch_bounds__(256) k_build_batch(const gnnshap::SolveJob* __restrict__ jobs) {
  const gnnshap::SolveJob J = jobs[blockIdx.y];
  if (blockIdx.x >= J.M || J.counts_in) return;
  build_row(reinterpret_cast<float*>(J.counts), J.usum, J.M, J.ld, J.kr > 0, J.alpha, J.wr, J.scal, blockIdx.x);
}

// One workgroup per job.
__global__ void __launch_bounds__(kMidThreads) k_solve_one_batch(const gnnshap::SolveJob* __restrict__ jobs) {
  const gnnshap::SolveJob J = jobs[blockIdx.x];
  if (J.panel) return;
  solve_mid_body(reinterpret_cast<float*>(J.counts), J.ld, J.M, J.dv, J.fef, J.Wd, J.info, J.phi);
}

// ---- panel path (kPanelMin < M <= kMidMax): one launch per panel step -----------------------
//
// The same blocked factorisation as the one-workgroup path (64-wide panels,
// diagonal factors inverted, L_Ip = A_Ip W_pp^T), spread over many small
// workgroups, one launch per panel: one workgroup per trailing tile (I, J)
// subtracts L_Ip L_Jp^T; the one holding the next diagonal block factors and
// inverts it, and each one in the next panel's column updates that diagonal
// block too, factors it again (the same operands and code, so the same
// bits) and forms its L_I,p+1 = A_I,p+1 W^T at once, so the next panel's
// blocks are ready when the launch ends.  The largest systems of a batch thus
// finish in ~20 us per panel instead of occupying one compute unit for their
// whole factorisation.  The
// factorisation reads G~ only, so it can run before the right-hand side
// exists; one workgroup per system then centres the right-hand side and runs
// the forward and backward substitutions (k_pp_solve).

constexpr size_t kPanelLds = (3 * kHB + 64) * sizeof(float);

// In LDS: D (lower part valid) <- chol, W <- its inverse, for diagonal block
// p of a system of M players (rows past M become the identity); `info`
// receives a non-positive pivot (NULL: not reported).  Four wavefronts.
__device__ __forceinline__ void pp_factor_diag(float* D, float* W, int64_t M, int64_t p, int32_t* info) {
  const int tid = threadIdx.x;
  if (tid < 64 && p * 64 + tid >= M) D[tid * kHP + tid] = 1.f;
  __syncthreads();
  if ((tid >> 6) == 0) chol_inv64(D, W, nullptr, p * 64, info);
  __syncthreads();
}

// Diagonal block p already in D0 (lower part; rows and columns past M zero):
// D0 <- L_pp, D1 <- W_pp = L_pp^-1, W_pp stored to Wd[p].  L_pp itself is
// not stored: the substitutions use W_pp, and G's diagonal block keeps the
// value the next panel's column workgroups read while this one runs.
__device__ __forceinline__ void pp_diag(float* G, int64_t ld, int64_t M, int64_t p, float* D0, float* D1,
                                        float* __restrict__ Wd, int32_t* info) {
  (void)G;
  (void)ld;
  pp_factor_diag(D0, D1, M, p, info);
  for (int t = threadIdx.x; t < 64 * 64; t += 256) Wd[p * 4096 + t] = D1[(t >> 6) * kHP + (t & 63)];
}

// Block (bi, bj) (64 x 64 at rows 64 bi, columns 64 bj) of G into S, zero past M;
// all sixteen loads of a thread are in flight before the LDS stores.
__device__ __forceinline__ void pp_load(const float* G, int64_t ld, int64_t M, int64_t bi, int64_t bj, float* S,
                                        bool lower_only) {
  const int tid = threadIdx.x;
  float v[16];
#pragma unroll
  for (int q = 0; q < 16; ++q) {
    const int t = tid + 256 * q, r = t >> 6, c = t & 63;
    const int64_t gi = 64 * bi + r, gj = 64 * bj + c;
    const bool ok = gi < M && gj < M && (!lower_only || c <= r);
    v[q] = ok ? G[gi * ld + gj] : 0.f;
  }
#pragma unroll
  for (int q = 0; q < 16; ++q) {
    const int t = tid + 256 * q;
    S[(t >> 6) * kHP + (t & 63)] = v[q];
  }
}

// Block bi of column p: A (in LDS, = A_{bi,p} updated by the earlier panels)
// <- L_{bi,p} = A W_pp^T, stored to G.
__device__ __forceinline__ void pp_form_column(float* G, int64_t ld, int64_t M, int64_t bi, int64_t p, float* A,
                                               const float* W) {
  mm64<true>(A, W, A, 1.f, 0.f);
  for (int t = threadIdx.x; t < 64 * 64; t += 256) {
    const int r = t >> 6, c = t & 63;
    if (64 * bi + r < M) G[(64 * bi + r) * ld + p * 64 + c] = A[r * kHP + c];
  }
}

// pp_load for a block that still holds the integer counts (the panel path's
// first touch of each block when G~ was not built in place): each entry is
// built on the way (gt_entry).
__device__ __forceinline__ void pp_load_counts(const gnnshap::SolveJob& J, int64_t bi, int64_t bj, float* S,
                                               bool lower_only) {
  const int tid = threadIdx.x;
  const int64_t M = J.M;
  const GtBuild b = gt_build(M, J.kr > 0, J.alpha, J.wr, J.scal);
  const int32_t* C = J.counts;
  int32_t cv[16];
  int64_t ui[16], uj[16];
#pragma unroll
  for (int q = 0; q < 16; ++q) {
    const int t = tid + 256 * q, r = t >> 6, c = t & 63;
    const int64_t gi = 64 * bi + r, gj = 64 * bj + c;
    const bool ok = gi < M && gj < M && (!lower_only || c <= r);
    cv[q] = (ok && b.has_random) ? C[gi * J.ld + gj] : 0;
    ui[q] = (ok && b.has_random) ? J.usum[gi] : 0;
    uj[q] = (ok && b.has_random) ? J.usum[gj] : 0;
  }
#pragma unroll
  for (int q = 0; q < 16; ++q) {
    const int t = tid + 256 * q, r = t >> 6, c = t & 63;
    const int64_t gi = 64 * bi + r, gj = 64 * bj + c;
    const bool ok = gi < M && gj < M && (!lower_only || c <= r);
    S[r * kHP + c] = ok ? gt_entry(b, cv[q], ui[q], uj[q], gi == gj) : 0.f;
  }
}

// A block of G~ as the panel path reads it: from the counts on a block's first
// touch when the system was not built in place, else as stored.
__device__ __forceinline__ void pp_load_g(const gnnshap::SolveJob& J, int64_t bi, int64_t bj, float* S,
                                          bool lower_only, bool first_touch) {
  if (first_touch && J.counts_in)
    pp_load_counts(J, bi, bj, S, lower_only);
  else
    pp_load(reinterpret_cast<const float*>(J.counts), J.ld, J.M, bi, bj, S, lower_only);
}

// Start, workgroup I of the first column: I = 0 factors diagonal block 0
// (info <- 0 first; L_00 and W_00 stored); I > 0 factors it too (not
// reported) and forms L_I0.
__device__ __forceinline__ void pp_start_body(const gnnshap::SolveJob& J, int64_t I) {
  extern __shared__ __align__(16) unsigned char smem[];
  float* D0 = reinterpret_cast<float*>(smem);
  float* D1 = D0 + kHB;
  float* A = D1 + kHB;
  float* G = reinterpret_cast<float*>(J.counts);
  const int64_t M = J.M, nblk = (M + 63) / 64;
  if (I >= nblk) return;
  if (I == 0) {
    if (threadIdx.x == 0) *J.info = 0;
    pp_load_g(J, 0, 0, D0, true, true);
    pp_diag(G, J.ld, M, 0, D0, D1, J.Wd, J.info);
    return;
  }
  pp_load_g(J, 0, 0, D0, true, true);
  pp_load_g(J, I, 0, A, false, true);
  pp_factor_diag(D0, D1, M, 0, nullptr);
  pp_form_column(G, J.ld, M, I, 0, A, D1);
}

// Panel p, trailing tile number `tile` (I >= J, row-major over the lower
// triangle of the blocks below panel p): A_IJ -= L_Ip L_Jp^T.  Tile (0, 0)
// is the next diagonal block and is factored at once (stored, reported);
// tiles (I, 0) update the next diagonal block as well, factor it and form
// L_{I, p+1}.
__device__ __forceinline__ void pp_trail_body(const gnnshap::SolveJob& J, int64_t p, int64_t tile) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int64_t M = J.M, nblk = (M + 63) / 64, nI = nblk - p - 1;
  // (a batched launch covers the batch's largest system: past this system's
  // last panel nI <= 0, and nI (nI + 1) / 2 is positive again for nI <= -2)
  if (nI <= 0 || tile >= nI * (nI + 1) / 2) return;
  int64_t I = 0;
  while ((I + 1) * (I + 2) / 2 <= tile) ++I;
  const int64_t Jb = tile - I * (I + 1) / 2;
  float* A = reinterpret_cast<float*>(smem);
  float* X = A + kHB;
  float* Y = X + kHB;
  float* G = reinterpret_cast<float*>(J.counts);
  const int tid = threadIdx.x;
  const int64_t bi = p + 1 + I, bj = p + 1 + Jb;
  pp_load_g(J, bi, bj, A, I == Jb, p == 0);
  pp_load(G, J.ld, M, bi, p, X, false);
  if (I != Jb) pp_load(G, J.ld, M, bj, p, Y, false);
  __syncthreads();
  mm64<true>(X, I == Jb ? X : Y, A, -1.f, 1.f);
  if (I == 0 && Jb == 0) {
    pp_diag(G, J.ld, M, p + 1, A, X, J.Wd, J.info);
    return;
  }
  if (Jb == 0) {
    // the next diagonal block: X <- A_{bj,bj} - L_{bj,p} L_{bj,p}^T, factored
    pp_load_g(J, bj, bj, X, true, p == 0);
    __syncthreads();
    mm64<true>(Y, Y, X, -1.f, 1.f);
    pp_factor_diag(X, Y, M, bj, nullptr);
    pp_form_column(G, J.ld, M, bi, bj, A, Y);
    return;
  }
  for (int t = tid; t < 64 * 64; t += 256) {
    const int r = t >> 6, c = t & 63;
    const int64_t gi = 64 * bi + r, gj = 64 * bj + c;
    if (gi < M && gj < M && (I != Jb || c <= r)) G[gi * J.ld + gj] = A[r * kHP + c];
  }
}

// One workgroup per system, after the factorisation and the right-hand
// side: r = P dv (centred, fp32), forward substitution z_p = W_pp (r_p -
// sum_{J<p} L_pJ z_J) panel by panel (left-looking: 16 threads per row read
// the row's L blocks), backward substitution psi_p = W_pp^T (z_p - sum_{I>p}
// L_Ip^T psi_I), phi = Delta/M + psi.  1024 threads, vectors in LDS.
constexpr int kBackThreads = 1024;

__device__ __forceinline__ void pp_solve_body(const gnnshap::SolveJob& J) {
  __shared__ float red[kBackThreads];
  __shared__ float vec[kMidMax];
  __shared__ float Wl[64 * 65];                  // W_pp of the current panel
  __shared__ double dred[kBackThreads / 64];
  const int64_t M = J.M, ld = J.ld, nblk = (M + 63) / 64;
  const float* G = reinterpret_cast<const float*>(J.counts);
  const int tid = threadIdx.x, c = tid & 63, g = tid >> 6;
  constexpr int NG = kBackThreads / 64;
  // centring: the mean of dv summed in a fixed order
  {
    double sv = 0.0;
    for (int64_t i = tid; i < M; i += kBackThreads) sv += J.dv[i];
    for (int off = 32; off > 0; off >>= 1) sv += __shfl_xor(sv, off);
    if (c == 0) dred[g] = sv;
    __syncthreads();
    double tot = 0.0;
#pragma unroll
    for (int gg = 0; gg < NG; ++gg) tot += dred[gg];
    const double mean = tot / static_cast<double>(M);
    for (int64_t i = tid; i < M; i += kBackThreads) vec[i] = static_cast<float>(J.dv[i] - mean);
    __syncthreads();
  }
  // forward: thread (r = tid / 16, q = tid % 16) of row o + r; rows r >= 64 idle
  {
    const int r = tid >> 4, q = tid & 15;
    for (int64_t p = 0; p < nblk; ++p) {
      const int64_t o = p * 64;
      float acc = 0.f;
      if (r < 64 && o + r < M) {
        const float* Lr = G + (o + r) * ld;
#pragma unroll 4
        for (int64_t col = q; col < o; col += 16) acc += Lr[col] * vec[col];
      }
      float wv[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) wv[e] = r < 64 ? J.Wd[p * 4096 + r * 64 + q + 16 * e] : 0.f;
#pragma unroll
      for (int off = 8; off > 0; off >>= 1) acc += __shfl_xor(acc, off, 16);
      if (r < 64 && q == 0) red[r] = o + r < M ? vec[o + r] - acc : 0.f;   // r_p - sum_J L_pJ z_J
      __syncthreads();
      float z = 0.f;
      if (r < 64) {
#pragma unroll
        for (int e = 0; e < 4; ++e) z += wv[e] * red[q + 16 * e];
      }
#pragma unroll
      for (int off = 8; off > 0; off >>= 1) z += __shfl_xor(z, off, 16);
      __syncthreads();
      if (r < 64 && q == 0 && o + r < M) vec[o + r] = z;
      __syncthreads();
    }
  }
  // backward
  for (int64_t p = nblk - 1; p >= 0; --p) {
    const int64_t o = p * 64;
    float wv[4096 / kBackThreads];
#pragma unroll
    for (int q = 0; q < 4096 / kBackThreads; ++q) wv[q] = J.Wd[p * 4096 + tid + kBackThreads * q];
    float acc = 0.f;
    if (o + c < M) {
#pragma unroll 4
      for (int64_t row = o + 64 + g; row < M; row += NG) acc += G[row * ld + o + c] * vec[row];
    }
    red[g * 64 + c] = acc;
#pragma unroll
    for (int q = 0; q < 4096 / kBackThreads; ++q) {
      const int t = tid + kBackThreads * q;
      Wl[(t >> 6) * 65 + (t & 63)] = wv[q];
    }
    __syncthreads();
    float t = 0.f;
    if (tid < 64) {
      float sum = 0.f;
#pragma unroll
      for (int gg = 0; gg < NG; ++gg) sum += red[gg * 64 + tid];
      t = o + tid < M ? vec[o + tid] - sum : 0.f;
    }
    __syncthreads();
    if (tid < 64) red[tid] = t;
    __syncthreads();
    if (tid < 64) {
      float ps = 0.f;
#pragma unroll 8
      for (int cc = tid; cc < 64; ++cc) ps += Wl[cc * 65 + tid] * red[cc];
      if (o + tid < M) vec[o + tid] = ps;
    }
    __syncthreads();
  }
  const double delta = static_cast<double>(J.fef[1]) - static_cast<double>(J.fef[0]);
  const double Md = static_cast<double>(M);
  for (int64_t i = tid; i < M; i += kBackThreads) J.phi[i] = static_cast<float>(delta / Md + static_cast<double>(vec[i]));
}

__global__ void __launch_bounds__(256) k_pp_start(const gnnshap::SolveJob* __restrict__ jobs) {
  const gnnshap::SolveJob J = jobs[blockIdx.y];
  if (J.panel) pp_start_body(J, blockIdx.x);
}
__global__ void __launch_bounds__(256) k_pp_trail(const gnnshap::SolveJob* __restrict__ jobs, int64_t p) {
  const gnnshap::SolveJob J = jobs[blockIdx.y];
  if (J.panel) pp_trail_body(J, p, blockIdx.x);
}
__global__ void __launch_bounds__(kBackThreads) k_pp_solve(const gnnshap::SolveJob* __restrict__ jobs) {
  const gnnshap::SolveJob J = jobs[blockIdx.x];
  if (J.panel) pp_solve_body(J);
}
__global__ void __launch_bounds__(256) k_pp_start_one(gnnshap::SolveJob J) { pp_start_body(J, blockIdx.x); }
__global__ void __launch_bounds__(256) k_pp_trail_one(gnnshap::SolveJob J, int64_t p) {
  pp_trail_body(J, p, blockIdx.x);
}
__global__ void __launch_bounds__(kBackThreads) k_pp_solve_one(gnnshap::SolveJob J) { pp_solve_body(J); }

// Whether `kernel` may be launched with `bytes` of dynamic LDS on the current
// device (its static LDS counts against the same limit); above the 64 KiB
// default, its dynamic limit is raised once to all the device allows.
bool allow_lds(const void* kernel, size_t bytes, bool& raised) {
  hipFuncAttributes a{};
  if (hipFuncGetAttributes(&a, kernel) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  const size_t cap = static_cast<size_t>(gnnshap::max_lds_bytes());
  const size_t fixed = a.sharedSizeBytes;
  if (bytes + fixed > cap) return false;
  if (bytes + fixed <= 65536) return true;
  if (!raised) {
    raised = hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                                 static_cast<int>(cap - fixed)) == hipSuccess;
    (void)hipGetLastError();
  }
  return raised;
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

namespace {

// Whether a factored system of M players is solved by one workgroup (its
// system in LDS) rather than by the multi-block Cholesky.
bool takes_mid(int64_t M) {
  static bool mid_lds = false;
  return M <= kMidMax && allow_lds(reinterpret_cast<const void*>(&k_solve_mid), kMidLds, mid_lds);
}

}  // namespace

// gnnshap_solve_wls up to the iteration of an iterative solve, whose system
// joins *grp (its set-up queued on the group's stream, which must be
// `stream`); other systems are queued in full and grp is left as it was.
int gnnshap::solve_wls_start(const gnnshap_sample_plan* plan, const gnnshap_class* classes, const uint64_t* masks,
                             const float* y, const float* f_empty_full, float* phi, int32_t* info, void* ws,
                             size_t ws_bytes, void* stream, CgGroup* grp, bool set_up_only) {
  GS_TRY_BEGIN
  gnnshap::clear_error();
  if (!classes || !masks || !y || !f_empty_full || !phi || !info || !ws)
    return gnnshap::fail(GNNSHAP_EINVAL, "null argument");
  if (int st = check_plan(plan, classes)) return st;
  gnnshap::Carver need(nullptr);
  carve(need, plan, classes);
  if (ws_bytes < need.bytes()) return gnnshap::fail(GNNSHAP_ECAPACITY, "solve workspace needs %zu bytes", need.bytes());
  gnnshap::Carver cv(ws);
  const Ws w = carve(cv, plan, classes);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t M = plan->num_players;
  const int64_t ld = ld_of(M);
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
  if (iterative(plan)) {
    if (set_up_only) return gnnshap::fail(GNNSHAP_EINVAL, "only a multi-block system is set up alone");
    // R as bit-transposed rows (the product R p), the right-hand side, then
    // conjugate gradients straight from the bits
    if (has_random) {
      GS_TIMED("k_transpose", s);
      k_transpose_blocked<<<dim3(static_cast<unsigned>(gnnshap::ceil_div(kr, 64)),
                                 static_cast<unsigned>(gnnshap::ceil_div(wpr, 8))),
                            512, 0, s>>>(masks, wpr, rb0, kr, M, w.T, w.cg.blocked);
    }
    GS_LAUNCHED();
    // the right-hand side: the enumerated rows from the row-major masks, the
    // random rows from their bit-transposed copy, then the chunks in order
    const int64_t nch_e = rhs_enum_chunks(plan);
    const int64_t nch_r = has_random ? rhs_rand_chunks(plan) : 0;
    k_dz<<<static_cast<unsigned>(gnnshap::ceil_div(half, 256)), 256, 0, s>>>(y, half, M, w.classes, plan->num_classes,
                                                                             f_empty_full, w.dz);
    GS_LAUNCHED();
    if (nch_e > 0) {
      GS_TIMED("k_rhs_part", s);
      const int64_t rpc = gnnshap::ceil_div(rb0, nch_e);
      k_rhs_part<<<dim3(static_cast<unsigned>(gnnshap::ceil_div(wpr, 4)), static_cast<unsigned>(nch_e)), 256, 0, s>>>(
          masks, wpr, rb0, M, w.dz, rpc, w.part);
    }
    GS_LAUNCHED();
    if (nch_r > 0) {
      const int64_t nxb = gnnshap::ceil_div(wpr, 8);
      if (nxb * nch_r > INT32_MAX) return gnnshap::fail(GNNSHAP_EUNSUPPORTED, "right-hand side grid too large");
      GS_TIMED("k_rhs_rand", s);
      k_rhs_rand<<<static_cast<unsigned>(nxb * nch_r), 512, 0, s>>>(w.T, M, wpr, kr, gnnshap::ceil_div(kr, 64),
                                                                    w.dz + rb0, w.part + nch_e * M, nxb);
    }
    GS_LAUNCHED();
    const int64_t nbm = gnnshap::ceil_div(M, 256);
    k_rhs_reduce<<<static_cast<unsigned>(nbm), 256, 0, s>>>(w.part, nch_e + nch_r, M, w.dv, w.bsum);
    GS_LAUNCHED();
    gnnshap::CgProblem pr{};
    pr.T = w.T;
    pr.blocked = w.cg.blocked;
    pr.dv = w.dv;
    pr.bsum = w.bsum;
    pr.nb = nbm;
    pr.classes = w.classes;
    pr.ncls = plan->num_classes;
    pr.rb0 = rb0;
    pr.alpha = alpha;
    pr.wr = wr;
    pr.fef = f_empty_full;
    pr.phi = phi;
    pr.info = info;
    if (grp->stream() != s) return gnnshap::fail(GNNSHAP_EINVAL, "solver group is on another stream");
    return grp->add(pr, cg_shape_of(plan, classes), w.cg);
  }
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
      k_gram<<<dim3(nb, nb), 256, 0, s>>>(w.T, nrb, M, ld, counts);
    }
    GS_LAUNCHED();
  }
  const bool mid = takes_mid(M);
  if (set_up_only && mid) return gnnshap::fail(GNNSHAP_EINVAL, "only a multi-block system is set up alone");
  const bool tiled = mid && rhs_tiled(M, plan->num_classes);
  const int64_t nch = tiled ? tile_chunks(half) : n_chunks(half, wpr);
  if (tiled) {
    GS_TIMED("k_rhs_tile", s);
    k_rhs_tile<<<static_cast<unsigned>(nch), kTileRows, 0, s>>>(masks, wpr, half, M, y, w.classes,
                                                               plan->num_classes, f_empty_full, w.part);
  } else {
    const int64_t rpc = gnnshap::ceil_div(half, nch);
    k_dz<<<static_cast<unsigned>(gnnshap::ceil_div(half, 256)), 256, 0, s>>>(y, half, M, w.classes,
                                                                             plan->num_classes, f_empty_full, w.dz);
    GS_LAUNCHED();
    GS_TIMED("k_rhs_part", s);
    k_rhs_part<<<dim3(static_cast<unsigned>(gnnshap::ceil_div(wpr, 4)), static_cast<unsigned>(nch)), 256, 0, s>>>(
        masks, wpr, half, M, w.dz, rpc, w.part);
  }
  GS_LAUNCHED();

  if (mid) {
    if (has_random) {
      k_rowsum<<<static_cast<unsigned>(gnnshap::ceil_div(M * 64, 256)), 256, 0, s>>>(counts, M, ld, w.usum);
      GS_LAUNCHED();
    }
    k_scalars<<<1, 256, 0, s>>>(counts, w.usum, M, ld, has_random, alpha, wr, f_empty_full, w.scal);
    GS_LAUNCHED();
    k_build<<<static_cast<unsigned>(M), 256, 0, s>>>(w.G, w.usum, M, ld, has_random, alpha, wr, w.scal);
    GS_LAUNCHED();
    const int64_t nbm = gnnshap::ceil_div(M, 256);
    k_rhs_reduce<<<static_cast<unsigned>(nbm), 256, 0, s>>>(w.part, nch, M, w.dv, w.bsum);
    GS_LAUNCHED();
    if (gnnshap::solve_panel_path(plan)) {
      gnnshap::SolveJob J{};
      J.panel = 1;
      J.counts = counts;
      J.ld = ld;
      J.M = M;
      J.dv = w.dv;
      J.rv = w.rhs;
      J.Wd = w.Wd;
      J.fef = f_empty_full;
      J.phi = phi;
      J.info = info;
      const int64_t nblk = gnnshap::ceil_div(M, 64);
      {
        GS_TIMED("k_pp_start", s);
        k_pp_start_one<<<static_cast<unsigned>(nblk), 256, kPanelLds, s>>>(J);
      }
      GS_LAUNCHED();
      for (int64_t p = 0; p + 1 < nblk; ++p) {
        const int64_t nI = nblk - p - 1;
        {
          GS_TIMED("k_pp_trail", s);
          k_pp_trail_one<<<static_cast<unsigned>(nI * (nI + 1) / 2), 256, kPanelLds, s>>>(J, p);
        }
        GS_LAUNCHED();
      }
      {
        GS_TIMED("k_pp_solve", s);
        k_pp_solve_one<<<1, kBackThreads, 0, s>>>(J);
      }
      GS_LAUNCHED();
      return GNNSHAP_OK;
    }
    {
      GS_TIMED("k_solve_mid", s);
      k_solve_mid<<<1, kMidThreads, kMidLds, s>>>(w.G, ld, M, w.dv, f_empty_full, w.Wd, info, phi);
    }
    GS_LAUNCHED();
    return GNNSHAP_OK;
  }

  static bool potrf_lds = false, fwd_lds = false, bwd_lds = false;
  if (!allow_lds(reinterpret_cast<const void*>(&k_potrf), kPotrfLds, potrf_lds) ||
      !allow_lds(reinterpret_cast<const void*>(&k_trsv_fwd), kTrsvLds, fwd_lds) ||
      !allow_lds(reinterpret_cast<const void*>(&k_trsv_bwd), kTrsvLds, bwd_lds))
    return gnnshap::fail(GNNSHAP_EHIP, "device cannot give the solver %zu bytes of LDS", kTrsvLds);
  k_zero_info<<<1, 1, 0, s>>>(info);
  GS_LAUNCHED();
  if (has_random) {
    k_rowsum<<<static_cast<unsigned>(gnnshap::ceil_div(M * 64, 256)), 256, 0, s>>>(counts, M, ld, w.usum);
    GS_LAUNCHED();
  }
  k_scalars<<<1, 256, 0, s>>>(counts, w.usum, M, ld, has_random, alpha, wr, f_empty_full, w.scal);
  GS_LAUNCHED();
  k_build<<<static_cast<unsigned>(M), 256, 0, s>>>(w.G, w.usum, M, ld, has_random, alpha, wr, w.scal);
  GS_LAUNCHED();
  const int64_t nbm = gnnshap::ceil_div(M, 256);
  k_rhs_reduce<<<static_cast<unsigned>(nbm), 256, 0, s>>>(w.part, nch, M, w.dv, w.bsum);
  GS_LAUNCHED();
  k_rhs_center<<<static_cast<unsigned>(nbm), 256, 0, s>>>(w.dv, w.bsum, nbm, M, w.rhs);
  GS_LAUNCHED();
  if (set_up_only) return GNNSHAP_OK;   // the rest runs batched (launch_solve_mb)
  for (int64_t o = 0; o < M; o += kPB) {
    {
      GS_TIMED("k_potrf", s);
      k_potrf<<<1, 256, kPotrfLds, s>>>(w.G, ld, M, o, info, w.Winv);
    }
    GS_LAUNCHED();
    const int64_t r0 = o + kPB;
    if (r0 >= M) break;
    const int64_t rows = M - r0;
    const int64_t tr = gnnshap::ceil_div(rows, kGT);
    float* panel = w.G + r0 * ld + o;
    {
      GS_TIMED("k_trsm", s);   // panel <- panel L_jj^-T = panel Winv^T
      k_gemm_nt<false><<<static_cast<unsigned>(tr), 256, 0, s>>>(panel, ld, w.Winv, kPB, panel, ld, rows, kPB, kPB,
                                                                  1.f, 0.f, 1);
    }
    GS_LAUNCHED();
    {
      GS_TIMED("k_syrk", s);   // trailing lower triangle -= panel panel^T
      k_gemm_nt<true><<<static_cast<unsigned>(tr * (tr + 1) / 2), 256, 0, s>>>(panel, ld, panel, ld, w.G + r0 * ld + r0,
                                                                                ld, rows, rows, kPB, -1.f, 1.f, 0);
    }
    GS_LAUNCHED();
  }
  // L x = rhs, L^T psi = x (psi into rhs), phi = Delta/M + psi
  for (int64_t s0 = 0; s0 < M; s0 += kSeg) {
    const int64_t s1 = std::min(M, s0 + kSeg);
    {
      GS_TIMED("k_trsv", s);
      k_trsv_fwd<<<1, 1024, kTrsvLds, s>>>(w.G, ld, s0, s1, w.rhs, w.x);
    }
    GS_LAUNCHED();
    if (s1 < M) {
      k_gemv_fwd<<<static_cast<unsigned>(gnnshap::ceil_div((M - s1) * 64, 256)), 256, 0, s>>>(w.G, ld, M, s0, s1, w.x,
                                                                                             w.rhs);
      GS_LAUNCHED();
    }
  }
  for (int64_t s0 = ((M - 1) / kSeg) * kSeg; s0 >= 0; s0 -= kSeg) {
    const int64_t s1 = std::min(M, s0 + kSeg);
    {
      GS_TIMED("k_trsv", s);
      k_trsv_bwd<<<1, 1024, kTrsvLds, s>>>(w.G, ld, s0, s1, w.x, w.rhs);
    }
    GS_LAUNCHED();
    if (s0 > 0) {
      k_gemv_bwd<<<static_cast<unsigned>(gnnshap::ceil_div(s0, 64)), 256, 0, s>>>(w.G, ld, s0, s1, w.rhs, w.x);
      GS_LAUNCHED();
    }
  }
  k_finish<<<gnnshap::grid_for(M, 256, 1024), 256, 0, s>>>(w.rhs, M, w.scal, phi);
  GS_LAUNCHED();
  return GNNSHAP_OK;
  GS_TRY_END
}

extern "C" int gnnshap_solve_wls(const gnnshap_sample_plan* plan, const gnnshap_class* classes,
                                 const uint64_t* masks, const float* y, const float* f_empty_full, float* phi,
                                 int32_t* info, void* ws, size_t ws_bytes, void* stream) {
  GS_TRY_BEGIN
  gnnshap::CgGroup grp;
  grp.set_stream(static_cast<hipStream_t>(stream));
  if (int st = gnnshap::solve_wls_start(plan, classes, masks, y, f_empty_full, phi, info, ws, ws_bytes, stream, &grp))
    return st;
  while (!grp.empty())
    if (int st = grp.step()) return st;
  return GNNSHAP_OK;
  GS_TRY_END
}

// ---- multi-target path: host side --------------------------------------------------------

bool gnnshap::solve_batchable(const gnnshap_sample_plan* plan) {
  if (check_plan(plan, nullptr) != GNNSHAP_OK) {
    clear_error();
    return false;
  }
  return plan->num_players <= kMidMax && rhs_tiled(plan->num_players, plan->num_classes) && !iterative(plan);
}

size_t gnnshap::solve_slice_bytes(const gnnshap_sample_plan* plan) {
  Carver c(nullptr);
  carve(c, plan);
  return c.bytes();
}

int gnnshap::solve_fill_job(const gnnshap_sample_plan* plan, const gnnshap_class* classes, void* slice,
                            SolveJob* job) {
  if (int st = check_plan(plan, classes)) return st;
  Carver c(slice);
  const Ws w = carve(c, plan);
  const int64_t M = plan->num_players;
  job->ncls = plan->num_classes;
  job->M = M;
  job->wpr = plan->words_per_row;
  job->half = plan->num_rows / 2;
  job->rb0 = plan->random_begin;
  job->kr = job->half - job->rb0;
  job->nrb = ceil_div(job->kr, 64);
  job->ld = ld_of(M);
  job->nch = tile_chunks(job->half);      // batched systems have at most kMidMax players
  job->wr = job->kr > 0 ? plan->random_weight : 0.0;
  double alpha = 0.0;
  for (int64_t i = 0; i < plan->num_classes; ++i) {
    if (!classes[i].full) continue;
    const int64_t cs = classes[i].size;
    const double kappa = 2 * cs < M ? 2.0 : 1.0;
    alpha += classes[i].weight * kappa * binom_d(M - 2, cs - 1);
  }
  job->alpha = alpha;
  job->T = w.T;
  job->counts = reinterpret_cast<int32_t*>(w.G);
  job->dz = w.dz;
  job->part = w.part;
  job->usum = w.usum;
  job->dv = w.dv;
  job->Wd = w.Wd;
  job->rv = w.rhs;
  job->panel = solve_panel_path(plan) ? 1 : 0;
  job->counts_in = job->panel;          // panel systems build G~ as their blocks are first read
  job->scal = w.scal;
  return GNNSHAP_OK;
}

bool gnnshap::solve_panel_path(const gnnshap_sample_plan* plan) {
  return solve_batchable(plan) && plan->num_players > kPanelMin;
}

bool gnnshap::solve_multiblock(const gnnshap_sample_plan* plan) {
  if (check_plan(plan, nullptr) != GNNSHAP_OK) {
    clear_error();
    return false;
  }
  return !iterative(plan) && !takes_mid(plan->num_players);
}

int gnnshap::solve_fill_mb_job(const gnnshap_sample_plan* plan, const gnnshap_class* classes, void* slice,
                               MbJob* job) {
  if (int st = check_plan(plan, classes)) return st;
  if (!solve_multiblock(plan)) return fail(GNNSHAP_EINVAL, "system does not take the multi-block path");
  Carver c(slice);
  const Ws w = carve(c, plan, classes);
  job->G = w.G;
  job->Winv = w.Winv;
  job->rhs = w.rhs;
  job->x = w.x;
  job->scal = w.scal;
  job->ld = ld_of(plan->num_players);
  job->M = plan->num_players;
  return GNNSHAP_OK;
}

int gnnshap::launch_solve_mb(const MbJob* jobs, int64_t n, int64_t max_M, hipStream_t s) {
  if (n < 1) return GNNSHAP_OK;
  if (n > 65535) return fail(GNNSHAP_EUNSUPPORTED, "at most 65535 multi-block systems per launch");
  static bool potrf_lds = false, fwd_lds = false, bwd_lds = false;
  if (!allow_lds(reinterpret_cast<const void*>(&k_potrf_mb), kPotrfLds, potrf_lds) ||
      !allow_lds(reinterpret_cast<const void*>(&k_trsv_fwd_mb), kTrsvLds, fwd_lds) ||
      !allow_lds(reinterpret_cast<const void*>(&k_trsv_bwd_mb), kTrsvLds, bwd_lds))
    return fail(GNNSHAP_EHIP, "device cannot give the solver %zu bytes of LDS", kTrsvLds);
  const unsigned nn = static_cast<unsigned>(n);
  for (int64_t o = 0; o < max_M; o += kPB) {
    {
      GS_TIMED("k_potrf_mb", s);
      k_potrf_mb<<<dim3(1, nn), 256, kPotrfLds, s>>>(jobs, o);
    }
    GS_LAUNCHED();
    const int64_t r0 = o + kPB;
    if (r0 >= max_M) break;
    const int64_t tr = ceil_div(max_M - r0, kGT);
    {
      GS_TIMED("k_trsm_mb", s);
      k_trsm_mb<<<dim3(static_cast<unsigned>(tr), nn), 256, 0, s>>>(jobs, o);
    }
    GS_LAUNCHED();
    {
      GS_TIMED("k_syrk_mb", s);
      k_syrk_mb<<<dim3(static_cast<unsigned>(tr * (tr + 1) / 2), nn), 256, 0, s>>>(jobs, o);
    }
    GS_LAUNCHED();
  }
  for (int64_t s0 = 0; s0 < max_M; s0 += kSeg) {
    {
      GS_TIMED("k_trsv_mb", s);
      k_trsv_fwd_mb<<<dim3(1, nn), 1024, kTrsvLds, s>>>(jobs, s0);
    }
    GS_LAUNCHED();
    const int64_t s1 = std::min(max_M, s0 + kSeg);
    if (s1 < max_M) {
      k_gemv_fwd_mb<<<dim3(static_cast<unsigned>(ceil_div((max_M - s1) * 64, 256)), nn), 256, 0, s>>>(jobs, s0);
      GS_LAUNCHED();
    }
  }
  for (int64_t s0 = ((max_M - 1) / kSeg) * kSeg; s0 >= 0; s0 -= kSeg) {
    {
      GS_TIMED("k_trsv_mb", s);
      k_trsv_bwd_mb<<<dim3(1, nn), 1024, kTrsvLds, s>>>(jobs, s0);
    }
    GS_LAUNCHED();
    if (s0 > 0) {
      k_gemv_bwd_mb<<<dim3(static_cast<unsigned>(ceil_div(s0, 64)), nn), 256, 0, s>>>(jobs, s0);
      GS_LAUNCHED();
    }
  }
  k_finish_mb<<<dim3(grid_for(max_M, 256, 1024), nn), 256, 0, s>>>(jobs);
  GS_LAUNCHED();
  return GNNSHAP_OK;
}

int gnnshap::launch_solve_matrix(const SolveJob* jobs, int64_t n, int64_t max_M, int64_t max_wpr, int64_t max_nrb,
                                 int64_t n_items, hipStream_t s) {
  (void)max_wpr;
  if (n < 1) return GNNSHAP_OK;
  if (n > 65535) return fail(GNNSHAP_EUNSUPPORTED, "at most 65535 targets per batch");
  const unsigned nn = static_cast<unsigned>(n);
  if (max_nrb > 0 && n_items > 0) {
    if (ceil_div(n_items, kTrWaves) > INT32_MAX) return fail(GNNSHAP_EUNSUPPORTED, "transpose grid too large");
    {
      GS_TIMED("k_transpose_batch", s);
      k_transpose_batch<<<static_cast<unsigned>(ceil_div(n_items, kTrWaves)), kTrWaves * 64, 0, s>>>(jobs, n, n_items);
    }
    GS_LAUNCHED();
    const int64_t nb = ceil_div(max_M, 64);
    {
      GS_TIMED("k_gram_batch", s);
      k_gram_batch<<<dim3(static_cast<unsigned>(nb * (nb + 1) / 2), static_cast<unsigned>(ceil_div(max_nrb, kGramChunk)),
                          nn),
                     256, 0, s>>>(jobs);
    }
    GS_LAUNCHED();
  }
  k_scalars_batch<<<nn, 256, 0, s>>>(jobs);
  GS_LAUNCHED();
  return GNNSHAP_OK;
}

int gnnshap::launch_solve_build(const SolveJob* jobs, int64_t n, int64_t max_M, hipStream_t s) {
  if (n < 1) return GNNSHAP_OK;
  if (n > 65535) return fail(GNNSHAP_EUNSUPPORTED, "at most 65535 targets per batch");
  k_build_batch<<<dim3(static_cast<unsigned>(max_M), static_cast<unsigned>(n)), 256, 0, s>>>(jobs);
  GS_LAUNCHED();
  return GNNSHAP_OK;
}

int gnnshap::launch_solve_rhs(const SolveJob* jobs, int64_t n, int64_t max_M, int64_t max_wpr, int64_t max_half,
                              int64_t max_nch, hipStream_t s) {
  if (n < 1) return GNNSHAP_OK;
  if (n > 65535) return fail(GNNSHAP_EUNSUPPORTED, "at most 65535 targets per batch");
  const unsigned nn = static_cast<unsigned>(n);
  {
    GS_TIMED("k_rhs_tile_batch", s);
    k_rhs_tile_batch<<<dim3(static_cast<unsigned>(max_nch), nn), kTileRows, 0, s>>>(jobs);
  }
  GS_LAUNCHED();
  k_rhs_sum_batch<<<dim3(static_cast<unsigned>(ceil_div(max_M, 256)), nn), 256, 0, s>>>(jobs);
  GS_LAUNCHED();
  return GNNSHAP_OK;
}

int gnnshap::launch_panel_factor(const SolveJob* jobs, int64_t n, int64_t max_panels, hipStream_t s) {
  if (n < 1 || max_panels < 1) return GNNSHAP_OK;
  if (n > 65535) return fail(GNNSHAP_EUNSUPPORTED, "at most 65535 targets per batch");
  const unsigned nn = static_cast<unsigned>(n);
  {
    GS_TIMED("k_pp_start", s);
    k_pp_start<<<dim3(static_cast<unsigned>(max_panels), nn), 256, kPanelLds, s>>>(jobs);
  }
  GS_LAUNCHED();
  for (int64_t p = 0; p + 1 < max_panels; ++p) {
    const int64_t nI = max_panels - p - 1;
    {
      GS_TIMED("k_pp_trail", s);
      k_pp_trail<<<dim3(static_cast<unsigned>(nI * (nI + 1) / 2), nn), 256, kPanelLds, s>>>(jobs, p);
    }
    GS_LAUNCHED();
  }
  return GNNSHAP_OK;
}

int gnnshap::launch_panel_solve(const SolveJob* jobs, int64_t n, hipStream_t s) {
  if (n < 1) return GNNSHAP_OK;
  if (n > 65535) return fail(GNNSHAP_EUNSUPPORTED, "at most 65535 targets per batch");
  GS_TIMED("k_pp_solve", s);
  k_pp_solve<<<static_cast<unsigned>(n), kBackThreads, 0, s>>>(jobs);
  GS_LAUNCHED();
  return GNNSHAP_OK;
}

int gnnshap::launch_solve_one(const SolveJob* jobs, int64_t n, hipStream_t s) {
  if (n < 1) return GNNSHAP_OK;
  if (n > 65535) return fail(GNNSHAP_EUNSUPPORTED, "at most 65535 targets per batch");
  const size_t lds = kMidLds;
  static bool raised = false;
  if (!allow_lds(reinterpret_cast<const void*>(&k_solve_one_batch), lds, raised))
    return fail(GNNSHAP_EUNSUPPORTED, "batched solve needs %zu bytes of LDS", lds);
  GS_TIMED("k_solve_one_batch", s);
  k_solve_one_batch<<<static_cast<unsigned>(n), kMidThreads, lds, s>>>(jobs);
  GS_LAUNCHED();
  return GNNSHAP_OK;
}

extern "C" int gnnshap_solve_info(const gnnshap_sample_plan* plan, int32_t* path) {
  gnnshap::clear_error();
  if (!path) return gnnshap::fail(GNNSHAP_EINVAL, "path is NULL");
  if (int st = check_plan(plan, nullptr)) return st;
  const int64_t M = plan->num_players;
  *path = iterative(plan) ? 3 : M > kMidMax ? 0 : (gnnshap::solve_panel_path(plan) ? 2 : 1);
  return GNNSHAP_OK;
}
