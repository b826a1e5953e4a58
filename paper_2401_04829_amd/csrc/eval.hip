// Masked GCN predictions for a batch of coalitions (Sec. 3.4 of the GNNShap
// paper; the GCN of Sec. 4.2).
//
// Layer l of the GCN under coalition S, at a node x within l-1 hops of v:
//   H^l[x] = act( d_x^-1/2 ( sum_{(u->x) in S} d_u^-1/2 Z^l[u] + d_x^-1/2 Z^l[x] ) + b_l ),
//   Z^l = H^(l-1) W_l,  d = 1 + in-degree under S.
// Only what reaches the target is computed: layer l is needed at the nodes
// within L-l hops.  Nodes at the computational graph's outer boundary (dist
// = hops) have no players entering them, so their representations do not
// depend on S; they are computed once per target ("constant" rows), as is
// Z^1 = X[V_c] W_1.  Everything else is per coalition:
//   degrees   popcount of the mask bits of each destination's player range;
//   aggregate a tile of 32 coalitions x one destination x a feature slice
//             per block: the constant source rows of a chunk of 64 players
//             are staged in LDS once and reused by all 32 coalitions;
//   transform (L >= 3) the per-coalition rows times W_l;
//   final     the target's logit, y = d_v^-1/2 (sum d_u^-1/2 H[u].w + d_v^-1/2 H[v].w) + b.
// Coalitions without an in-edge of v are not evaluated (Sec. 3.4.1): their
// value is f(empty), which is exact.  f(empty) and f(E_c) come from two extra
// rows (no players / all players) run through the same kernels first.
#include "batch.h"
#include "common.h"
#include "wide.h"

namespace {

constexpr int kTB = 32;          // coalitions per aggregation block
constexpr int kChunkE = 64;      // players staged per step
constexpr size_t kTileBudget = size_t(1) << 30;  // bytes of per-coalition scratch

struct Shape {
  int L = 0, hops = 0;
  int64_t n_nodes = 0, n_dst = 0, bnd0 = 0, bnd1 = 0;  // boundary rows [bnd0, bnd1)
  int dims[GNNSHAP_MAX_LAYERS + 1] = {};
  int64_t nd[GNNSHAP_MAX_LAYERS + 1] = {};  // rows of H^j that depend on S: [0, nd[j])
  bool bnd[GNNSHAP_MAX_LAYERS + 1] = {};    // H^j is needed at the boundary rows
  int64_t tile = 0;                          // coalitions per pass
  int64_t k = 0, wpr = 0;
  bool wide = false;                         // two layers, two hops, wide hidden layer: eval_wide.hip
  gnnshap::WideShape ws;
};

struct Ws {
  int32_t* ctl;        // [0] class, [1] live count
  uint64_t* sp_masks;  // 2 rows: no players, all players
  int32_t* sp_rows;    // {0, 1}
  float* sp_y;         // 2 x C
  int32_t* live_rows;  // k
  uint8_t* live_flag;  // k
  float* Zc[GNNSHAP_MAX_LAYERS + 1];  // constant Z^j rows (n_nodes x dims[j])
  float* Bc[GNNSHAP_MAX_LAYERS + 1];  // constant H^j rows at the boundary
  float* dinv;                        // tile x n_dst
  float* Hb[GNNSHAP_MAX_LAYERS + 1];  // tile x nd[j] x dims[j]
  float* Zb[GNNSHAP_MAX_LAYERS + 1];  // tile x nd[j-1] x dims[j]
  gnnshap::WideWs wide;               // the wide path's arrays (Shape::wide)
};

int64_t per_row_bytes(const Shape& s) {
  int64_t b = s.n_dst;
  for (int j = 1; j < s.L; ++j) b += s.nd[j] * s.dims[j];
  for (int j = 2; j < s.L; ++j) b += s.nd[j - 1] * s.dims[j];
  return 4 * b;
}

Ws carve(gnnshap::Carver& c, const Shape& s) {
  Ws w{};
  const int C = s.dims[s.L];
  w.ctl = c.take<int32_t>(8);
  w.sp_masks = c.take<uint64_t>(2 * s.wpr);
  w.sp_rows = c.take<int32_t>(2);
  w.sp_y = c.take<float>(2 * C);
  w.live_rows = c.take<int32_t>(s.k);
  w.live_flag = c.take<uint8_t>(s.k);
  w.Zc[1] = c.take<float>(s.n_nodes * s.dims[1]);
  for (int j = 1; j < s.L; ++j) {
    if (!s.bnd[j]) continue;
    w.Bc[j] = c.take<float>(s.n_nodes * s.dims[j]);
    if (j + 1 < s.L) w.Zc[j + 1] = c.take<float>(s.n_nodes * s.dims[j + 1]);
  }
  w.dinv = c.take<float>(s.tile * s.n_dst);
  for (int j = 1; j < s.L; ++j) w.Hb[j] = c.take<float>(s.tile * s.nd[j] * s.dims[j]);
  for (int j = 2; j < s.L; ++j) w.Zb[j] = c.take<float>(s.tile * s.nd[j - 1] * s.dims[j]);
  if (s.wide) w.wide = gnnshap::wide_carve(c, s.ws);
  return w;
}

int make_shape(const gnnshap_subgraph* sg, const gnnshap_gcn* m, int64_t k, Shape* out) {
  if (!sg || !m || !m->dims) return gnnshap::fail(GNNSHAP_EINVAL, "null subgraph or model");
  Shape s;
  s.L = m->num_layers;
  s.hops = sg->num_hops;
  if (s.L < 1 || s.L > GNNSHAP_MAX_LAYERS) return gnnshap::fail(GNNSHAP_EINVAL, "num_layers out of range");
  if (s.hops < 1 || s.hops > GNNSHAP_MAX_HOPS) return gnnshap::fail(GNNSHAP_EINVAL, "num_hops out of range");
  for (int j = 0; j <= s.L; ++j) {
    s.dims[j] = m->dims[j];
    if (s.dims[j] < 1 || s.dims[j] > (1 << 20)) return gnnshap::fail(GNNSHAP_EINVAL, "bad layer width");
  }
  if (s.dims[s.L] > GNNSHAP_MAX_CLASSES) return gnnshap::fail(GNNSHAP_EUNSUPPORTED, "too many classes");
  s.n_nodes = sg->num_nodes;
  s.n_dst = sg->num_dst;
  if (s.n_nodes < 1 || s.n_dst < 1 || s.n_dst > s.n_nodes || sg->hop_ptr[s.hops] != s.n_dst ||
      sg->hop_ptr[s.hops + 1] != s.n_nodes || sg->num_edges < 1)
    return gnnshap::fail(GNNSHAP_EINVAL, "subgraph sizes are inconsistent");
  s.bnd0 = sg->hop_ptr[s.hops];
  s.bnd1 = sg->hop_ptr[s.hops + 1];
  s.nd[0] = 0;
  for (int j = 1; j <= s.L; ++j) {
    const int r = std::min(s.L - j, s.hops - 1);
    s.nd[j] = sg->hop_ptr[r + 1];
    s.bnd[j] = (s.L - j) >= s.hops && s.bnd1 > s.bnd0;
  }
  s.k = k;
  s.wpr = (sg->num_edges + 63) / 64;
  const int64_t prb = per_row_bytes(s);
  int64_t t = static_cast<int64_t>(kTileBudget / static_cast<size_t>(prb > 0 ? prb : 1));
  if (t >= k) t = k;                 // one pass covers every row
  else if (t >= kTB) t -= t % kTB;
  if (t < 2) t = 2;
  s.tile = t;
  // The wide path evaluates every row in a launch sequence of its own; the
  // per-pass arrays above then serve the two end coalitions only.
  s.wide = gnnshap::wide_applies(s.L, s.hops, s.dims);
  if (s.wide) {
    s.tile = 2;
    s.ws = gnnshap::wide_shape(sg->num_edges, s.n_nodes, s.n_dst, sg->hop_ptr[2], k, s.dims, s.L);
  }
  *out = s;
  return GNNSHAP_OK;
}

__device__ __forceinline__ int64_t rows_in_pass(const int32_t* dyn_count, int64_t dyn_off, int64_t cap) {
  if (!dyn_count) return cap;
  int64_t r = static_cast<int64_t>(*dyn_count) - dyn_off;
  return r < 0 ? 0 : (r > cap ? cap : r);
}

__global__ void k_init(int32_t* ctl, uint64_t* sp_masks, int32_t* sp_rows, int64_t wpr, int64_t M) {
  const int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (t < 8) ctl[t] = 0;
  if (t < 2) sp_rows[t] = static_cast<int32_t>(t);
  for (int64_t w = t; w < wpr; w += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    sp_masks[w] = 0;
    const int64_t lo = w * 64;
    const int64_t nb = M - lo >= 64 ? 64 : M - lo;
    sp_masks[wpr + w] = nb >= 64 ? ~uint64_t(0) : ((uint64_t(1) << nb) - 1);
  }
}

typedef float mx4_t __attribute__((ext_vector_type(4)));

// C[m, :] = op(A[row(m), :]) B for m in [m0, m0 + rows), 64x64 tiles, fp32
// MFMA (16x16x4) with fp32 accumulation.  row(m) = arow ? arow[m] : m;
// op(a) = relu(a + abias) if abias else a.  The 16-wide K slices are staged
// in LDS; the next one is fetched into registers while the current one is
// multiplied.
__global__ void __launch_bounds__(256) k_gemm(const float* __restrict__ A, int64_t lda,
                                              const int32_t* __restrict__ arow,
                                              const float* __restrict__ abias,
                                              const float* __restrict__ B, int64_t ldb,
                                              float* __restrict__ C, int64_t ldc, int64_t m0,
                                              int64_t rows, int64_t N, int64_t K,
                                              const int32_t* dyn_count, int64_t dyn_off,
                                              int64_t dyn_cap, int64_t dyn_mult) {
  // row stride 80: the 4 x 16 operand reads of a wavefront hit 64 distinct banks
  __shared__ float As[16][80];
  __shared__ float Bs[16][80];
  if (dyn_count) {
    const int64_t r = rows_in_pass(dyn_count, dyn_off, dyn_cap) * dyn_mult;
    if (r < rows) rows = r;
  }
  const int64_t mb = m0 + static_cast<int64_t>(blockIdx.x) * 64;
  if (mb >= m0 + rows) return;
  const int64_t nb = static_cast<int64_t>(blockIdx.y) * 64;
  const int tid = threadIdx.x;
  const int kk = tid % 16, kb0 = tid / 64, nn = tid % 64;
  const float* arp[4];
  bool aok[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t m = mb + tid / 16 + 16 * i;
    aok[i] = m < m0 + rows;
    const int64_t ar = aok[i] ? (arow ? static_cast<int64_t>(arow[m]) : m) : 0;
    arp[i] = A + ar * lda;
  }
  const bool nok = nb + nn < N;
  float ra[4], rb[4];
  auto fetch = [&](int64_t k0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float a = 0.f;
      if (aok[i] && k0 + kk < K) {
        a = arp[i][k0 + kk];
        if (abias) a = fmaxf(a + abias[k0 + kk], 0.f);
      }
      ra[i] = a;
      const int64_t kr = k0 + kb0 + 4 * i;
      rb[i] = (kr < K && nok) ? B[kr * ldb + nb + nn] : 0.f;
    }
  };
  // wavefront w multiplies rows 16 w .. 16 w + 15 of the tile by its 64
  // columns on fp32 MFMA (16x16x4): lane (r, g) = (lane % 16, lane / 16)
  // gives A[16 w + r][k + g] and B[k + g][16 nt + r], and holds D rows
  // 16 w + 4 g .. + 3 of column 16 nt + r
  const int wave = tid >> 6, lane = tid & 63, r = lane & 15, g = lane >> 4;
  mx4_t acc[4];
#pragma unroll
  for (int nt = 0; nt < 4; ++nt) acc[nt] = mx4_t{0.f, 0.f, 0.f, 0.f};
  fetch(0);
  for (int64_t k0 = 0; k0 < K; k0 += 16) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      As[kk][tid / 16 + 16 * i] = ra[i];
      Bs[kb0 + 4 * i][nn] = rb[i];
    }
    __syncthreads();
    if (k0 + 16 < K) fetch(k0 + 16);
#pragma unroll
    for (int q = 0; q < 16; q += 4) {
      const float av = As[q + g][16 * wave + r];
#pragma unroll
      for (int nt = 0; nt < 4; ++nt)
        acc[nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, Bs[q + g][16 * nt + r], acc[nt], 0, 0, 0);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t m = mb + 16 * wave + 4 * g + i;
    if (m >= m0 + rows) continue;
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) {
      const int64_t n = nb + 16 * nt + r;
      if (n < N) C[m * ldc + n] = acc[nt][i];
    }
  }
}

// Zc[u, :] = XW1[node_gid[u], :]
__global__ void k_gather_rows(const float* __restrict__ src, const int32_t* __restrict__ idx, int64_t n, int h,
                              float* __restrict__ dst) {
  const int64_t total = n * h;
  for (int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; t < total;
       t += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const int64_t u = t / h, f = t % h;
    dst[t] = src[static_cast<int64_t>(idx[u]) * h + f];
  }
}

__global__ void k_bias_relu(const float* __restrict__ Z, const float* __restrict__ bias,
                            float* __restrict__ H, int64_t r0, int64_t r1, int h) {
  const int64_t total = (r1 - r0) * h;
  for (int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; t < total;
       t += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const int64_t idx = r0 * h + t;
    const float bb = bias ? bias[t % h] : 0.f;
    H[idx] = fmaxf(Z[idx] + bb, 0.f);
  }
}

// dinv[b, x] = (1 + popcount of row b's bits in player range of x)^-1/2.
__global__ void __launch_bounds__(256) k_degrees(const uint64_t* __restrict__ masks, int64_t wpr,
                                                 const int32_t* __restrict__ rows, int64_t row_off,
                                                 int64_t cap, const int32_t* dyn_count,
                                                 const int32_t* __restrict__ dst_ptr, int64_t n_dst,
                                                 float* __restrict__ dinv) {
  const int64_t nr = rows_in_pass(dyn_count, row_off, cap);
  const int64_t total = nr * n_dst;
  for (int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; t < total;
       t += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const int64_t b = t / n_dst, x = t % n_dst;
    const uint64_t* mrow = masks + static_cast<int64_t>(rows[row_off + b]) * wpr;
    const int64_t e0 = dst_ptr[x], e1 = dst_ptr[x + 1];
    int cnt = 0;
    for (int64_t w = e0 >> 6; w <= ((e1 - 1) >> 6) && e1 > e0; ++w) {
      uint64_t word = mrow[w];
      const int64_t lo = w * 64;
      if (e0 > lo) word &= ~uint64_t(0) << (e0 - lo);
      if (e1 < lo + 64) word &= (uint64_t(1) << (e1 - lo)) - 1;
      cnt += __popcll(word);
    }
    dinv[t] = rsqrtf(1.0f + static_cast<float>(cnt));
  }
}

// Masked aggregation of layer j for a tile of kTB coalitions, one destination
// x and one feature slice of width 8*FPT.  Thread (tb, fg): coalition tb,
// features fs0 + fg*FPT .. +FPT.
template <int FPT>
__global__ void __launch_bounds__(256) k_aggregate(
    const uint64_t* __restrict__ masks, int64_t wpr, const int32_t* __restrict__ rows,
    int64_t row_off, int64_t cap, const int32_t* dyn_count, const int32_t* __restrict__ dst_ptr,
    const int32_t* __restrict__ edge_src, int64_t n_dst, const float* __restrict__ dinv,
    const float* __restrict__ Zc, const float* __restrict__ Zb, int64_t nd_prev,
    const float* __restrict__ bias, float* __restrict__ Hout, int64_t nd_out, int h,
    int64_t n_tiles, int n_slices) {
  constexpr int FS = 8 * FPT;
  __shared__ float zs[kChunkE][FS];
  __shared__ int32_t ss[kChunkE];
  const int64_t nr = rows_in_pass(dyn_count, row_off, cap);
  int64_t bid = blockIdx.x;
  const int slice = static_cast<int>(bid % n_slices);
  bid /= n_slices;
  const int64_t tile = bid % n_tiles;
  const int64_t x = bid / n_tiles;
  if (tile * kTB >= nr) return;
  const int tid = threadIdx.x;
  const int tb = tid >> 3, fg = tid & 7;
  const int64_t b = tile * kTB + tb;
  const bool valid = b < nr;
  const int fs0 = slice * FS;
  const int f0 = fs0 + fg * FPT;
  const uint64_t* mrow = valid ? masks + static_cast<int64_t>(rows[row_off + b]) * wpr : masks;
  const float* drow = dinv + (valid ? b : 0) * n_dst;
  const float* zbrow = Zb ? Zb + (valid ? b : 0) * nd_prev * h : nullptr;
  float acc[FPT];
#pragma unroll
  for (int i = 0; i < FPT; ++i) acc[i] = 0.f;
  const int64_t e0 = dst_ptr[x], e1 = dst_ptr[x + 1];
  for (int64_t ec = e0; ec < e1; ec += kChunkE) {
    const int n = static_cast<int>(e1 - ec < kChunkE ? e1 - ec : kChunkE);
    if (tid < n) ss[tid] = edge_src[ec + tid];
    __syncthreads();
    for (int idx = tid; idx < n * FS; idx += 256) {
      const int e = idx / FS, f = idx % FS;
      const int32_t u = ss[e];
      zs[e][f] = (u >= nd_prev && fs0 + f < h) ? Zc[static_cast<int64_t>(u) * h + fs0 + f] : 0.f;
    }
    uint64_t bits = 0;
    if (valid) {
      const int64_t w0 = ec >> 6;
      const int sh = static_cast<int>(ec & 63);
      bits = mrow[w0] >> sh;
      if (sh && w0 + 1 < wpr) bits |= mrow[w0 + 1] << (64 - sh);
      if (n < 64) bits &= (uint64_t(1) << n) - 1;
    }
    __syncthreads();
    while (bits) {
      const int e = __ffsll(static_cast<long long>(bits)) - 1;
      bits &= bits - 1;
      const int32_t u = ss[e];
      const float coef = u < n_dst ? drow[u] : 1.0f;
      if (u < nd_prev) {
        const float* zr = zbrow + static_cast<int64_t>(u) * h;
#pragma unroll
        for (int i = 0; i < FPT; ++i)
          if (f0 + i < h) acc[i] += coef * zr[f0 + i];
      } else {
#pragma unroll
        for (int i = 0; i < FPT; ++i) acc[i] += coef * zs[e][fg * FPT + i];
      }
    }
    __syncthreads();
  }
  if (!valid) return;
  const float dx = drow[x];
  const float* zx = x < nd_prev ? zbrow + x * h : Zc + x * h;
  float* out = Hout + (b * nd_out + x) * h;
#pragma unroll
  for (int i = 0; i < FPT; ++i) {
    const int f = f0 + i;
    if (f < h) {
      const float v = dx * (acc[i] + dx * zx[f]) + (bias ? bias[f] : 0.f);
      out[f] = fmaxf(v, 0.f);
    }
  }
}

// The target's logit for each coalition of the pass: one wavefront per row.
// T(u) = u < nd_last ? Hb[b, u] : Hc[u] (width h); y = d_v^-1/2 (sum_{S} d_u^-1/2
// T(u).w_c + d_v^-1/2 T(v).w_c) + b_c.  With one layer T(u).w_c = Z^1[u, c].
__global__ void __launch_bounds__(256) k_final(
    const uint64_t* __restrict__ masks, int64_t wpr, const int32_t* __restrict__ rows,
    int64_t row_off, int64_t cap, const int32_t* dyn_count, const int32_t* __restrict__ dst_ptr,
    const int32_t* __restrict__ edge_src, int64_t n_dst, const float* __restrict__ dinv,
    const float* __restrict__ Hb, const float* __restrict__ Hc, int64_t nd_last, int h,
    const float* __restrict__ WL, const float* __restrict__ bL, int C, bool one_layer,
    const int32_t* __restrict__ ctl, bool all_classes, float* __restrict__ y_rows,
    float* __restrict__ y_all) {
  const int64_t nr = rows_in_pass(dyn_count, row_off, cap);
  const int lane = threadIdx.x & 63;
  const int64_t b = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) >> 6;
  if (b >= nr) return;
  const int64_t row = rows[row_off + b];
  const uint64_t* mrow = masks + row * wpr;
  const float* drow = dinv + b * n_dst;
  const float dv = drow[0];
  const int64_t e1 = dst_ptr[1];
  const int c_lo = all_classes ? 0 : ctl[0];
  const int c_hi = all_classes ? C : c_lo + 1;
  for (int c = c_lo; c < c_hi; ++c) {
    float acc = 0.f;
    for (int64_t e = 0; e < e1; ++e) {
      if (!((mrow[e >> 6] >> (e & 63)) & 1)) continue;
      const int32_t u = edge_src[e];
      const float coef = u < n_dst ? drow[u] : 1.0f;
      if (one_layer) {
        if (lane == 0) acc += coef * Hc[static_cast<int64_t>(u) * C + c];
      } else {
        const float* t = u < nd_last ? Hb + (b * nd_last + u) * h : Hc + static_cast<int64_t>(u) * h;
        float d = 0.f;
        for (int f = lane; f < h; f += 64) d += t[f] * WL[static_cast<int64_t>(f) * C + c];
        acc += coef * d;
      }
    }
    {
      if (one_layer) {
        if (lane == 0) acc += dv * Hc[c];
      } else {
        const float* t = 0 < nd_last ? Hb + (b * nd_last) * h : Hc;
        float d = 0.f;
        for (int f = lane; f < h; f += 64) d += t[f] * WL[static_cast<int64_t>(f) * C + c];
        acc += dv * d;
      }
    }
    for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
    const float yv = dv * acc + (bL ? bL[c] : 0.f);
    if (lane == 0) {
      if (all_classes) y_all[b * C + c] = yv;
      else y_rows[row] = yv;
    }
  }
}

// Two-layer GCN with hops >= 2, one launch per pass: a block takes `tbr` <=
// kTB coalitions and runs, in LDS,
//   degrees  dinv[b, x] for every destination x;
//   layer 1  at every x in H_1: masked aggregation of Z^1 = X W_1 rows
//            (staged 64 players at a time), ReLU, then t[b, x, c] =
//            H^1[b, x] . W_2[:, c] for the explained class (or every class);
//   layer 2  y = d_v^-1/2 (sum_{(u->v) in S} d_u^-1/2 t[u] + d_v^-1/2 t[v]) + b_2.
template <int FPT>
__device__ __forceinline__ void eval_l2_body(
    const uint64_t* __restrict__ masks, int64_t wpr, const int32_t* __restrict__ rows, int64_t row_off,
    int64_t cap, const int32_t* dyn_count, const int32_t* __restrict__ dst_ptr,
    const int32_t* __restrict__ edge_src, int64_t n_dst, int64_t n1, const float* __restrict__ Zc,
    const float* __restrict__ b1, const float* __restrict__ W2, const float* __restrict__ b2, int h, int C,
    const int32_t* __restrict__ ctl, bool all_classes, int tbr, float* __restrict__ y_rows,
    float* __restrict__ y_all, int64_t block) {
  constexpr int FS = 8 * FPT;
  extern __shared__ __align__(16) float sm[];
  const int ncls = all_classes ? C : 1;
  float* dinv = sm;                                   // tbr x n_dst
  float* tt = dinv + tbr * n_dst;                     // tbr x n1 x ncls
  float* zs = tt + tbr * n1 * ncls;                   // 64 x FS
  int32_t* ss = reinterpret_cast<int32_t*>(zs + kChunkE * FS);
  const int64_t nr = rows_in_pass(dyn_count, row_off, cap);
  const int64_t b_base = block * tbr;
  if (b_base >= nr) return;
  const int tid = threadIdx.x;
  const int tb = tid >> 3, fg = tid & 7;
  const int64_t b = b_base + tb;
  const bool valid = tb < tbr && b < nr;
  const uint64_t* mrow = valid ? masks + static_cast<int64_t>(rows[row_off + b]) * wpr : masks;
  const int c0 = all_classes ? 0 : ctl[0];

  // degrees
  for (int64_t t = tid; t < static_cast<int64_t>(tbr) * n_dst; t += 256) {
    const int64_t bb = t / n_dst, x = t % n_dst;
    float d = 1.0f;
    if (b_base + bb < nr) {
      const uint64_t* mr = masks + static_cast<int64_t>(rows[row_off + b_base + bb]) * wpr;
      const int64_t e0 = dst_ptr[x], e1 = dst_ptr[x + 1];
      int cnt = 0;
      for (int64_t w = e0 >> 6; e1 > e0 && w <= ((e1 - 1) >> 6); ++w) {
        uint64_t word = mr[w];
        const int64_t lo = w * 64;
        if (e0 > lo) word &= ~uint64_t(0) << (e0 - lo);
        if (e1 < lo + 64) word &= (uint64_t(1) << (e1 - lo)) - 1;
        cnt += __popcll(word);
      }
      d = rsqrtf(1.0f + static_cast<float>(cnt));
    }
    dinv[t] = d;
  }
  for (int64_t t = tid; t < static_cast<int64_t>(tbr) * n1 * ncls; t += 256) tt[t] = 0.f;
  __syncthreads();
  const float* drow = dinv + (valid ? tb : 0) * n_dst;

  // layer 1 at every node of H_1, folded into the class logits
  for (int64_t x = 0; x < n1; ++x) {
    const int64_t e0 = dst_ptr[x], e1 = dst_ptr[x + 1];
    const float dx = drow[x];
    for (int fs0 = 0; fs0 < h; fs0 += FS) {
      const int f0 = fs0 + fg * FPT;
      float acc[FPT];
#pragma unroll
      for (int i = 0; i < FPT; ++i) acc[i] = 0.f;
      for (int64_t ec = e0; ec < e1; ec += kChunkE) {
        const int n = static_cast<int>(e1 - ec < kChunkE ? e1 - ec : kChunkE);
        __syncthreads();
        if (tid < n) ss[tid] = edge_src[ec + tid];
        __syncthreads();
        for (int idx = tid; idx < n * FS; idx += 256) {
          const int e = idx / FS, f = idx % FS;
          zs[idx] = fs0 + f < h ? Zc[static_cast<int64_t>(ss[e]) * h + fs0 + f] : 0.f;
        }
        uint64_t bits = 0;
        if (valid) {
          const int64_t w0 = ec >> 6;
          const int sh = static_cast<int>(ec & 63);
          bits = mrow[w0] >> sh;
          if (sh && w0 + 1 < wpr) bits |= mrow[w0 + 1] << (64 - sh);
          if (n < 64) bits &= (uint64_t(1) << n) - 1;
        }
        __syncthreads();
        while (bits) {
          const int e = __ffsll(static_cast<long long>(bits)) - 1;
          bits &= bits - 1;
          const int32_t u = ss[e];
          const float coef = u < n_dst ? drow[u] : 1.0f;
#pragma unroll
          for (int i = 0; i < FPT; ++i) acc[i] += coef * zs[e * FS + fg * FPT + i];
        }
      }
      float hv[FPT];
#pragma unroll
      for (int i = 0; i < FPT; ++i) {
        const int f = f0 + i;
        hv[i] = f < h ? fmaxf(dx * (acc[i] + dx * Zc[x * h + f]) + (b1 ? b1[f] : 0.f), 0.f) : 0.f;
      }
      for (int ci = 0; ci < ncls; ++ci) {
        float p = 0.f;
#pragma unroll
        for (int i = 0; i < FPT; ++i)
          if (f0 + i < h) p += hv[i] * W2[static_cast<int64_t>(f0 + i) * C + c0 + ci];
        p += __shfl_xor(p, 1);
        p += __shfl_xor(p, 2);
        p += __shfl_xor(p, 4);
        if (valid && fg == 0) tt[(tb * n1 + x) * ncls + ci] += p;
      }
    }
  }
  __syncthreads();

  // layer 2 at the target
  const int64_t indeg = dst_ptr[1];
  for (int t = tid; t < tbr * ncls; t += 256) {
    const int bb = t / ncls, ci = t % ncls;
    const int64_t bg = b_base + bb;
    if (bg >= nr) continue;
    const int64_t row = rows[row_off + bg];
    const uint64_t* mr = masks + row * wpr;
    const float* dr = dinv + bb * n_dst;
    const float dv = dr[0];
    float acc = 0.f;
    for (int64_t e = 0; e < indeg; ++e) {
      if (!((mr[e >> 6] >> (e & 63)) & 1)) continue;
      const int32_t u = edge_src[e];
      acc += dr[u] * tt[(bb * n1 + u) * ncls + ci];
    }
    acc += dv * tt[(bb * n1) * ncls + ci];
    const float yv = dv * acc + (b2 ? b2[c0 + ci] : 0.f);
    if (all_classes) y_all[bg * C + ci] = yv;
    else y_rows[row] = yv;
  }
}

// Z^1 row of local node u: Zsrc row zidx[u] (the graph-wide X W_1 and the
// subgraph's node ids), or row u when zidx is NULL (per-subgraph rows).
__device__ __forceinline__ const float* zrow(const float* __restrict__ Zsrc, const int32_t* __restrict__ zidx,
                                             int32_t u, int h) {
  return Zsrc + static_cast<int64_t>(zidx ? zidx[u] : u) * h;
}

// Main pass of the two-layer evaluation with one thread per coalition, for
// narrow hidden layers (h <= H): a block of kRowsPerBlock coalitions stages
// what they all read (each player's source and Z^1 row, Z^1 of H_1, the
// destinations' player ranges) in LDS once; per coalition the in-degrees of
// the destinations (16-bit counts in LDS), then layer 1 at every node x of
// H_1 folded into the explained logit and, as x goes, layer 2 at the target:
// node x >= 1 of H_1 is the source of the target's player x - 1 (local ids
// sort the in-neighbours by global id, as the players entering the target).
constexpr int kRowsPerBlock = 128;

// Row stride of the staged Z^1 rows: four floats of padding spread the
// coalitions' scattered row reads over the LDS banks.
constexpr int zstride(int H) { return H + 4; }

size_t rows_lds_bytes(int64_t n_dst, int64_t n1, int64_t M, int H) {
  return sizeof(float) * static_cast<size_t>(M * zstride(H) + n1 * H) +
         sizeof(uint16_t) * static_cast<size_t>(kRowsPerBlock * (n_dst + 1)) +
         sizeof(int32_t) * static_cast<size_t>(M + n_dst + 1) + 16;
}

template <int H>
__device__ __forceinline__ void eval_rows_body(
    const uint64_t* __restrict__ masks, int64_t wpr, const int32_t* __restrict__ rows, int64_t cap,
    const int32_t* dyn_count, const int32_t* __restrict__ dst_ptr, const int32_t* __restrict__ edge_src,
    int64_t n_dst, int64_t n1, int64_t M, const float* __restrict__ Zsrc, const int32_t* __restrict__ zidx,
    const float* __restrict__ b1, const float* __restrict__ W2, const float* __restrict__ b2, int h, int C,
    const int32_t* __restrict__ ctl, const float* __restrict__ fef, float* __restrict__ y_rows, int64_t block) {
  constexpr int R = kRowsPerBlock;
  constexpr int ZS = zstride(H);
  extern __shared__ __align__(16) float sm[];
  float* zall = sm;                                            // M x ZS
  float* zself = zall + M * ZS;                                // n1 x H
  int32_t* sall = reinterpret_cast<int32_t*>(zself + n1 * H);  // M: source, or n_dst past the destinations
  int32_t* dptr = sall + M;                                    // n_dst + 1
  uint16_t* deg = reinterpret_cast<uint16_t*>(dptr + n_dst + 1);  // (n_dst + 1) x R, row n_dst = 0
  const int64_t nr = rows_in_pass(dyn_count, 0, cap);
  const int64_t b0 = block * R;
  if (b0 >= nr) return;
  const int tid = threadIdx.x;
  const int64_t b = b0 + tid;
  const bool valid = b < nr;
  const int c0 = ctl[0];
  const int nd = static_cast<int>(n_dst), Mi = static_cast<int>(M), n1i = static_cast<int>(n1);
  // a source outside the destinations has no player entering it: degree 1,
  // coefficient rsqrt(1 + 0), read from the zero row n_dst
#pragma unroll 4
  for (int e = tid; e < Mi; e += R) {
    const int32_t u = edge_src[e];
    sall[e] = u < nd ? u : nd;
  }
  for (int x = tid; x <= nd; x += R) dptr[x] = dst_ptr[x];
#pragma unroll 4
  for (int t = tid; t < n1i * H; t += R) {
    const int x = t / H, f = t % H;
    zself[t] = f < h ? zrow(Zsrc, zidx, x, h)[f] : 0.f;
  }
  deg[nd * R + tid] = 0;
#pragma unroll 4
  for (int t = tid; t < Mi * H; t += R) {
    const int e = t / H, f = t % H;
    zall[e * ZS + f] = f < h ? zrow(Zsrc, zidx, edge_src[e], h)[f] : 0.f;
  }
  __syncthreads();
  const int64_t row = valid ? (rows ? static_cast<int64_t>(rows[b]) : b) : 0;
  const uint64_t* mrow = masks + row * wpr;
  // without a row list every row is taken; one with no player entering the
  // target is pruned: its value is f(empty) (Sec. 3.4.1)
  bool live = valid;
  if (!rows && valid) {
    const int indeg = dptr[1];
    bool any = false;
    for (int w = 0; w * 64 < indeg; ++w) {
      uint64_t word = mrow[w];
      if (indeg - w * 64 < 64) word &= (uint64_t(1) << (indeg - w * 64)) - 1;
      any = any || word != 0;
    }
    live = any;
    if (!live) y_rows[row] = fef[0];
  }
  // in-degree of every destination under this coalition
  for (int x = 0; x < nd && live; ++x) {
    const int e0 = dptr[x], e1 = dptr[x + 1];
    int cnt = 0;
    for (int w = e0 >> 6; e1 > e0 && w <= ((e1 - 1) >> 6); ++w) {
      uint64_t word = mrow[w];
      const int lo = w * 64;
      if (e0 > lo) word &= ~uint64_t(0) << (e0 - lo);
      if (e1 < lo + 64) word &= (uint64_t(1) << (e1 - lo)) - 1;
      cnt += __popcll(word);
    }
    deg[x * R + tid] = static_cast<uint16_t>(cnt);
  }
  float w2v[H], b1v[H];
#pragma unroll
  for (int i = 0; i < H; ++i) {
    w2v[i] = i < h ? W2[static_cast<int64_t>(i) * C + c0] : 0.f;
    b1v[i] = (b1 && i < h) ? b1[i] : 0.f;
  }
  __syncthreads();
  // 1 + deg >= 1: the hardware reciprocal square root needs no denormal scaling
  auto dinv = [&](int x) { return __builtin_amdgcn_rsqf(1.0f + static_cast<float>(deg[x * R + tid])); };
  // layer 1 at every node of H_1, folded into the explained logit; layer 2 alongside
  if (!live) return;
  float acc2 = 0.f, t0 = 0.f;
  for (int x = 0; x < n1i; ++x) {
    const int e0 = dptr[x], e1 = dptr[x + 1];
    float acc[H];
#pragma unroll
    for (int i = 0; i < H; ++i) acc[i] = 0.f;
    for (int w = e0 >> 6; e1 > e0 && w <= ((e1 - 1) >> 6); ++w) {
      uint64_t bits = mrow[w];
      const int lo = w * 64;
      if (e0 > lo) bits &= ~uint64_t(0) << (e0 - lo);
      if (e1 < lo + 64) bits &= (uint64_t(1) << (e1 - lo)) - 1;
      // the two 32-bit halves of the word, set bits in ascending order
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        uint32_t hb = static_cast<uint32_t>(bits >> (32 * half));
        const int base = lo + 32 * half;
        while (hb) {
          const int e = base + __builtin_ctz(hb);
          hb &= hb - 1;
          const float coef = dinv(sall[e]);
          const float* z = zall + __umul24(e, ZS);
#pragma unroll
          for (int i = 0; i < H; i += 4) {
            const float4 zz = *reinterpret_cast<const float4*>(z + i);
            acc[i] += coef * zz.x;
            acc[i + 1] += coef * zz.y;
            acc[i + 2] += coef * zz.z;
            acc[i + 3] += coef * zz.w;
          }
        }
      }
    }
    const float dx = dinv(x);
    float p = 0.f;
#pragma unroll
    for (int i = 0; i < H; ++i) {
      const float hv = i < h ? fmaxf(dx * (acc[i] + dx * zself[x * H + i]) + b1v[i], 0.f) : 0.f;
      p += hv * w2v[i];
    }
    if (x == 0) {
      t0 = p;
    } else if ((mrow[(x - 1) >> 6] >> ((x - 1) & 63)) & 1) {
      acc2 += dx * p;
    }
  }
  // layer 2 at the target
  const float dv = dinv(0);
  acc2 += dv * t0;
  y_rows[row] = dv * acc2 + (b2 ? b2[c0] : 0.f);
}

template <int H>
__global__ void __launch_bounds__(kRowsPerBlock) k_eval_rows(
    const uint64_t* __restrict__ masks, int64_t wpr, const int32_t* __restrict__ rows, int64_t cap,
    const int32_t* dyn_count, const int32_t* __restrict__ dst_ptr, const int32_t* __restrict__ edge_src,
    int64_t n_dst, int64_t n1, int64_t M, const float* __restrict__ Zsrc, const int32_t* __restrict__ zidx,
    const float* __restrict__ b1, const float* __restrict__ W2, const float* __restrict__ b2, int h, int C,
    const int32_t* __restrict__ ctl, const float* __restrict__ fef, float* __restrict__ y_rows) {
  eval_rows_body<H>(masks, wpr, rows, cap, dyn_count, dst_ptr, edge_src, n_dst, n1, M, Zsrc, zidx, b1, W2, b2, h, C,
                    ctl, fef, y_rows, blockIdx.x);
}

// The same pass for h <= 16 on fp32 MFMA.  Layer 1 at node x of H_1 under
// a coalition c is a contraction over the players entering x:
//   acc[f][c] = sum_e Z^1[src e][f] * coef[e][c],
//   coef[e][c] = [e in c] * d_c(src e)^-1/2,
// so a wavefront evaluates 64 coalitions as four 16 x 16 output tiles
// (features x coalitions) with v_mfma_f32_16x16x4f32, four players per step:
// A (16 features x 4 players) is the staged Z^1 rows, shared by the tiles,
// B (4 players x 16 coalitions) the mask bit ANDed into the bits of
// d^-1/2, which a first phase computes for every destination and coalition
// of the workgroup.  Per node, lane (rl, g) then holds features 4g..4g+3 of
// coalition rl of each tile: self loop, bias and ReLU are applied in
// registers and the result, weighted by the node's layer-2 coefficient, is
// accumulated per feature; the explained logit's weights and the sum over
// the four lane groups (two butterflies) come once, after the last node.
// Each coalition's value depends on its own column only, so a row gets the
// same value whichever rows share its workgroup.
constexpr int kMxRows = 256;             // coalitions per workgroup (4 wavefronts)
constexpr int kMxDvs = kMxRows + 16;     // row stride of the d^-1/2 table

size_t rows_mx_lds_bytes(int64_t n_dst, int64_t n1, int64_t M) {
  const int64_t nw = 2 * ((M + 63) / 64);
  return sizeof(float) * static_cast<size_t>((M + 8) * 16 + n1 * 16 + (n_dst + 1) * kMxDvs + (nw + 2) * kMxRows +
                                             (M + 8) + (n_dst + 1) + 2 * kMxRows);
}


__device__ __forceinline__ void eval_rows_mx_body(
    const uint64_t* __restrict__ masks, int64_t wpr, const int32_t* __restrict__ rows, int64_t cap,
    const int32_t* dyn_count, const int32_t* __restrict__ dst_ptr, const int32_t* __restrict__ edge_src,
    int64_t n_dst, int64_t n1, int64_t M, const float* __restrict__ Zsrc, const int32_t* __restrict__ zidx,
    const float* __restrict__ b1, const float* __restrict__ W2, const float* __restrict__ b2, int h, int C,
    const int32_t* __restrict__ ctl, const float* __restrict__ fef, float* __restrict__ y_rows, int64_t block) {
  constexpr int R = kMxRows, DVS = kMxDvs;
  extern __shared__ __align__(16) float sm[];
  const int Mi = static_cast<int>(M), nd = static_cast<int>(n_dst), n1i = static_cast<int>(n1);
  const int nw = static_cast<int>(2 * wpr);                            // 32-bit words per mask row
  float* zall = sm;                                                    // (M + 8) x 16: Z^1 of each player's source
  float* zself = zall + (Mi + 8) * 16;                                 // n1 x 16: Z^1 of H_1
  float* dv = zself + n1i * 16;                                        // (n_dst + 1) x DVS: d^-1/2, row n_dst = 1
  uint32_t* m32 = reinterpret_cast<uint32_t*>(dv + (nd + 1) * DVS);  // (nw + 2) x R: mask words, two zero rows
  int32_t* sall = reinterpret_cast<int32_t*>(m32 + (nw + 2) * R);     // M + 8: DVS x (source, or n_dst)
  int32_t* dptr = sall + Mi + 8;                                       // n_dst + 1
  int32_t* rowid = dptr + nd + 1;                                      // R
  int32_t* live = rowid + R;                                           // R
  const int64_t nr = rows_in_pass(dyn_count, 0, cap);
  const int64_t b0 = block * R;
  if (b0 >= nr) return;
  const int tid = threadIdx.x;
  const int c0 = ctl[0];
  for (int e = tid; e < Mi + 8; e += R) {
    const int32_t u = e < Mi ? edge_src[e] : nd;
    sall[e] = (u < nd ? u : nd) * DVS;
  }
  for (int x = tid; x <= nd; x += R) dptr[x] = dst_ptr[x];
  for (int t = tid; t < n1i * 16; t += R) {
    const int x = t >> 4, f = t & 15;
    zself[t] = f < h ? zrow(Zsrc, zidx, x, h)[f] : 0.f;
  }
#pragma unroll 4
  for (int t = tid; t < (Mi + 8) * 16; t += R) {
    const int e = t >> 4, f = t & 15;
    zall[t] = (e < Mi && f < h) ? zrow(Zsrc, zidx, edge_src[e], h)[f] : 0.f;
  }
  // phase 1, one thread per coalition: its row, mask words (transposed),
  // d^-1/2 of every destination, and whether any player enters the target
  const int64_t bi = b0 + tid;
  const bool valid = bi < nr;
  const int64_t row = valid ? (rows ? static_cast<int64_t>(rows[bi]) : bi) : 0;
  rowid[tid] = static_cast<int32_t>(row);
  {
    const uint64_t* mrow = masks + row * wpr;
    for (int j = 0; j < wpr; ++j) {
      const uint64_t word = valid ? mrow[j] : 0;
      m32[(2 * j) * R + tid] = static_cast<uint32_t>(word);
      m32[(2 * j + 1) * R + tid] = static_cast<uint32_t>(word >> 32);
    }
    m32[nw * R + tid] = 0;
    m32[(nw + 1) * R + tid] = 0;
  }
  __syncthreads();
  for (int x = 0; x < nd; ++x) {
    const int e0 = dptr[x], e1 = dptr[x + 1];
    int cnt = 0;
    for (int j = e0 >> 5; e1 > e0 && j <= ((e1 - 1) >> 5); ++j) {
      uint32_t word = m32[j * R + tid];
      const int lo = j * 32;
      if (e0 > lo) word &= ~0u << (e0 - lo);
      if (e1 < lo + 32) word &= (1u << (e1 - lo)) - 1;
      cnt += __popc(word);
    }
    if (x == 0) live[tid] = cnt > 0;
    // 1 + deg >= 1: the hardware reciprocal square root needs no denormal scaling
    dv[x * DVS + tid] = __builtin_amdgcn_rsqf(1.0f + static_cast<float>(cnt));
  }
  dv[nd * DVS + tid] = 1.0f;
  __syncthreads();
  // phase 2, one wavefront per 64 coalitions
  const int lane = tid & 63, rl = lane & 15, g = lane >> 4;
  const int cb = (tid & ~63) + rl;               // coalition of lane (rl, g) in tile t: cb + 16 t
  float b1v[4], w2v[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int f = 4 * g + r;
    b1v[r] = (b1 && f < h) ? b1[f] : 0.f;
    w2v[r] = f < h ? W2[static_cast<int64_t>(f) * C + c0] : 0.f;
  }
  float S[4][4];
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int r = 0; r < 4; ++r) S[t][r] = 0.f;
  for (int x = 0; x < n1i; ++x) {
    const int e0 = __builtin_amdgcn_readfirstlane(dptr[x]);
    const int e1 = __builtin_amdgcn_readfirstlane(dptr[x + 1]);
    const int ng = (e1 - e0 + 3) >> 2;           // steps of four players
    mx4_t D[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) D[t] = mx4_t{0.f, 0.f, 0.f, 0.f};
    for (int q0 = 0; q0 < ng; q0 += 8) {
      // lane (rl, g) takes players s, s + 4, ..., s + 28: one 32-bit window per tile
      const int s = e0 + 4 * q0 + g;
      const int j = s >> 5, sh = s & 31;
      uint32_t win[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const uint32_t lo = m32[j * R + cb + 16 * t], hi = m32[(j + 1) * R + cb + 16 * t];
        win[t] = static_cast<uint32_t>(((static_cast<uint64_t>(hi) << 32) | lo) >> sh);
      }
      const int nq = ng - q0 < 8 ? ng - q0 : 8;
      auto step = [&](int q, float a, const float* dvv) {
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const int bit = __builtin_amdgcn_sbfe(static_cast<int>(win[t]), 4 * q, 1);   // 0 or -1
          const float bv = __int_as_float(__float_as_int(dvv[t]) & bit);
          D[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, bv, D[t], 0, 0, 0);
        }
      };
      // two steps at a time: both steps' reads are issued before the first product
      int q = 0;
      for (; q + 1 < nq; q += 2) {
        const int ea = s + 4 * q, eb = ea + 4;
        const int ua = sall[ea], ub = sall[eb];
        const float za = zall[ea * 16 + rl], zb = zall[eb * 16 + rl];
        float da[4], db[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          da[t] = dv[ua + cb + 16 * t];
          db[t] = dv[ub + cb + 16 * t];
        }
        __builtin_amdgcn_sched_barrier(0);   // keep every read ahead of the products
        step(q, ea < e1 ? za : 0.f, da);
        step(q + 1, eb < e1 ? zb : 0.f, db);
      }
      if (q < nq) {
        const int ea = s + 4 * q;
        const int ua = sall[ea];
        const float za = zall[ea * 16 + rl];
        float da[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) da[t] = dv[ua + cb + 16 * t];
        step(q, ea < e1 ? za : 0.f, da);
      }
    }
    // H^1 at node x and its weight in layer 2 at the target: d_x^-1/2 when
    // node x is the target itself or the source of a player in the
    // coalition, else 0.  The explained logit is linear in these terms, so
    // S accumulates weight * H^1 per feature and the sum over features (the
    // four lane groups) is taken once at the end.
    const float4 zs = *reinterpret_cast<const float4*>(zself + x * 16 + 4 * g);
    const float zsv[4] = {zs.x, zs.y, zs.z, zs.w};
    const int xw = x > 0 ? ((x - 1) >> 5) * R : 0, xb = (x - 1) & 31;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int c = cb + 16 * t;
      const float dx = dv[x * DVS + c];
      const float wx = (x == 0 || ((m32[xw + c] >> xb) & 1)) ? dx : 0.f;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float hv = fmaxf(fmaf(dx, fmaf(dx, zsv[r], D[t][r]), b1v[r]), 0.f);
        S[t][r] = fmaf(wx, hv, S[t][r]);
      }
    }
  }
  // explained logit per coalition: sum over features, then layer 2's outer
  // d_target^-1/2 and bias; lane (rl, g) writes coalition rl of tile g, or
  // f(empty) when no player enters the target (Sec. 3.4.1)
  float pt[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    float p = 0.f;
#pragma unroll
    for (int r = 0; r < 4; ++r) p = fmaf(S[t][r], w2v[r], p);
    p += __shfl_xor(p, 16);
    p += __shfl_xor(p, 32);
    pt[t] = p;
  }
  float p = pt[0];
#pragma unroll
  for (int t = 1; t < 4; ++t)
    if (g == t) p = pt[t];
  const int c = cb + 16 * g;
  if (b0 + c < nr) {
    const float dv0 = dv[c];
    y_rows[rowid[c]] = (live[c] || !fef) ? fmaf(dv0, p, b2 ? b2[c0] : 0.f) : fef[0];
  }
}

__global__ void __launch_bounds__(kMxRows) k_eval_rows_mx(
    const uint64_t* __restrict__ masks, int64_t wpr, const int32_t* __restrict__ rows, int64_t cap,
    const int32_t* dyn_count, const int32_t* __restrict__ dst_ptr, const int32_t* __restrict__ edge_src,
    int64_t n_dst, int64_t n1, int64_t M, const float* __restrict__ Zsrc, const int32_t* __restrict__ zidx,
    const float* __restrict__ b1, const float* __restrict__ W2, const float* __restrict__ b2, int h, int C,
    const int32_t* __restrict__ ctl, const float* __restrict__ fef, float* __restrict__ y_rows) {
  eval_rows_mx_body(masks, wpr, rows, cap, dyn_count, dst_ptr, edge_src, n_dst, n1, M, Zsrc, zidx, b1, W2, b2, h, C,
                    ctl, fef, y_rows, blockIdx.x);
}

// The per-coalition main pass of a two-layer model (h <= 32): its LDS bytes,
// 0 when the target's shapes do not fit, and the coalitions per workgroup.
size_t rows_pass_lds(int64_t n_dst, int64_t n1, int64_t M, int h) {
  size_t b = 0;
  if (h <= 16) b = rows_mx_lds_bytes(n_dst, n1, M);
  else if (h <= 32) b = rows_lds_bytes(n_dst, n1, M, 32);
  return b <= 65536 ? b : 0;
}
int rows_pass_block(int h) { return h <= 16 ? kMxRows : kRowsPerBlock; }

__device__ __forceinline__ void pick_class(const float* __restrict__ sp_y, int C, int requested, int32_t* ctl,
                                           int32_t* class_out, float* f_empty_full) {
  int c = requested;
  if (c < 0) {
    c = 0;
    for (int i = 1; i < C; ++i)
      if (sp_y[C + i] > sp_y[C + c]) c = i;
  }
  ctl[0] = c;
  if (class_out) *class_out = c;
  f_empty_full[0] = sp_y[c];
  f_empty_full[1] = sp_y[C + c];
}

// The two end coalitions of a two-layer GCN with hops >= 2 (no players and
// every player), every class, in one workgroup: the full coalition's degrees
// are the in-degrees of the subgraph; layer 1 runs with one thread per
// (node of H_1, feature), the class logits per (node, class) and layer 2 per
// class.  sp_y[c] = f_c(empty), sp_y[C + c] = f_c(E_c).
constexpr int kEndsThreads = 256;

size_t ends_lds_bytes(int64_t n_dst, int64_t n1, int h, int C) {
  const int64_t nx = h >= kEndsThreads ? 1 : kEndsThreads / h;
  return sizeof(float) * static_cast<size_t>(n_dst + n1 * C + nx * h + h + C);
}

// Extra LDS when the workgroup keeps Z^1 of the subgraph (n_nodes x h), the
// players' sources (M), the node ids, the destinations' player ranges and
// W_2 in LDS: global memory is then read once, in two rounds of independent
// loads, and the per-node loops read LDS only.
size_t ends_stage_bytes(int64_t n_nodes, int64_t n_dst, int64_t M, int h, int C) {
  return sizeof(float) * static_cast<size_t>(n_nodes * h + M + n_nodes + n_dst + 1 + static_cast<int64_t>(h) * C);
}

// LDS of the end-coalition kernel, staged (S) when it fits in 64 KiB.
size_t ends_launch_lds(int64_t n_dst, int64_t n1, int64_t n_nodes, int64_t M, int h, int C, bool* S) {
  const size_t base = ends_lds_bytes(n_dst, n1, h, C);
  const size_t staged = base + ends_stage_bytes(n_nodes, n_dst, M, h, C);
  *S = staged <= 65536;
  return *S ? staged : base;
}

// With XW1 given, the workgroup first gathers Zc (n_nodes x h) = the rows of
// XW1 at the subgraph's node ids (for this kernel and the next ones);
// afterwards thread 0 picks the explained class (requested, or argmax
// f(E_c)) into ctl[0], class_out and f_empty_full.  The values do not depend
// on S (only where the operands are read from).
template <bool S>
__device__ __forceinline__ void ends_l2_body(const int32_t* __restrict__ dst_ptr,
                                             const int32_t* __restrict__ edge_src, int64_t n_dst, int64_t n1,
                                             int64_t M, float* Zc, const float* __restrict__ XW1,
                                             const int32_t* __restrict__ node_gid, int64_t n_nodes,
                                             const float* __restrict__ b1,
                                             const float* __restrict__ W2, const float* __restrict__ b2, int h,
                                             int C, float* __restrict__ sp_y, int requested, int32_t* ctl,
                                             int32_t* class_out, float* f_empty_full) {
  extern __shared__ __align__(16) float sm[];
  const int tid = threadIdx.x;
  const float* Zr = Zc;                 // operands as read below: global memory, or their LDS copies
  const int32_t* er = edge_src;
  const int32_t* dp = dst_ptr;
  const float* w2 = W2;
  float* rest = sm;
  if constexpr (S) {
    float* Zl = sm;                                                  // n_nodes x h
    int32_t* el = reinterpret_cast<int32_t*>(Zl + n_nodes * h);     // M
    int32_t* gl = el + M;                                            // n_nodes
    int32_t* dl = gl + n_nodes;                                      // n_dst + 1
    float* wl = reinterpret_cast<float*>(dl + n_dst + 1);           // h x C
    for (int64_t e = tid; e < M; e += kEndsThreads) el[e] = edge_src[e];
    if (XW1)
      for (int64_t i = tid; i < n_nodes; i += kEndsThreads) gl[i] = node_gid[i];
    for (int64_t x = tid; x <= n_dst; x += kEndsThreads) dl[x] = dst_ptr[x];
    for (int64_t i = tid; i < static_cast<int64_t>(h) * C; i += kEndsThreads) wl[i] = W2[i];
    __syncthreads();
    const bool vec = (h & 3) == 0 && (reinterpret_cast<uintptr_t>(Zc) & 15) == 0 &&
                     (!XW1 || (reinterpret_cast<uintptr_t>(XW1) & 15) == 0);
    if (vec) {
      // rows of four floats, eight loads in flight per thread
      const int hq = h >> 2;
      const int64_t total = n_nodes * hq;
      for (int64_t t0 = tid; t0 < total; t0 += 8 * kEndsThreads) {
        float4 v[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const int64_t t = t0 + q * kEndsThreads;
          if (t < total) {
            const int64_t i = t / hq, c4 = t % hq;
            v[q] = XW1 ? reinterpret_cast<const float4*>(XW1 + static_cast<int64_t>(gl[i]) * h)[c4]
                       : reinterpret_cast<const float4*>(Zc)[t];
          }
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const int64_t t = t0 + q * kEndsThreads;
          if (t < total) {
            reinterpret_cast<float4*>(Zl)[t] = v[q];
            if (XW1) reinterpret_cast<float4*>(Zc)[t] = v[q];
          }
        }
      }
    } else {
      const int64_t total = n_nodes * h;
      for (int64_t t0 = tid; t0 < total; t0 += 8 * kEndsThreads) {
        float v[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const int64_t t = t0 + q * kEndsThreads;
          v[q] = t < total ? (XW1 ? XW1[static_cast<int64_t>(gl[t / h]) * h + t % h] : Zc[t]) : 0.f;
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const int64_t t = t0 + q * kEndsThreads;
          if (t < total) {
            Zl[t] = v[q];
            if (XW1) Zc[t] = v[q];
          }
        }
      }
    }
    Zr = Zl;
    er = el;
    dp = dl;
    w2 = wl;
    rest = wl + static_cast<int64_t>(h) * C;
    __syncthreads();
  } else if (XW1) {
    const int64_t total = n_nodes * h;
    for (int64_t t0 = tid; t0 < total; t0 += 4 * kEndsThreads) {
      float v[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int64_t t = t0 + q * kEndsThreads;
        v[q] = t < total ? XW1[static_cast<int64_t>(node_gid[t / h]) * h + t % h] : 0.f;
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int64_t t = t0 + q * kEndsThreads;
        if (t < total) Zc[t] = v[q];
      }
    }
    __syncthreads();
  }
  const int64_t nx = h >= kEndsThreads ? 1 : kEndsThreads / h;
  float* dinv = rest;                 // n_dst: full-coalition d^-1/2
  float* tt = dinv + n_dst;           // n1 x C: H^1[x] . W_2[:, c] under the full coalition
  float* hv = tt + n1 * C;            // nx x h: H^1 rows of the current node chunk
  float* he = hv + nx * h;            // h: H^1 row of the target under the empty coalition
  float* te = he + h;                 // C
  for (int64_t x = tid; x < n_dst; x += kEndsThreads)
    dinv[x] = rsqrtf(1.0f + static_cast<float>(dp[x + 1] - dp[x]));
  const float d0 = rsqrtf(1.0f);      // degree factor of every node when no edge is present
  for (int f = tid; f < h; f += kEndsThreads)
    he[f] = fmaxf(d0 * (0.0f + d0 * Zr[f]) + (b1 ? b1[f] : 0.f), 0.f);
  __syncthreads();
  const int lane = tid & 63, wv = tid >> 6;
  // the class logits of the nodes of one chunk, from their H^1 rows in hv
  auto chunk_logits = [&](int64_t x0, int64_t nn) {
    for (int64_t it = tid; it < nn * C; it += kEndsThreads) {
      const int64_t xi = it / C;
      const int c = static_cast<int>(it % C);
      float t = 0.f;
      for (int f = 0; f < h; ++f) t += hv[xi * h + f] * w2[static_cast<int64_t>(f) * C + c];
      tt[(x0 + xi) * C + c] = t;
    }
  };
  if (h <= 16) {
    // one wavefront per node of H_1, four nodes at a time: lane (f, slot)
    // takes feature f of every fourth player from the slot on (four loads in
    // flight), and two butterflies add the four slots
    const int f = lane & 15, slot = lane >> 4;
    for (int64_t x0 = 0; x0 < n1; x0 += 4) {
      const int64_t nn = n1 - x0 < 4 ? n1 - x0 : 4;
      const int64_t x = x0 + wv;
      float acc = 0.f;
      if (x < n1 && f < h) {
        const int64_t e0 = dp[x], e1 = dp[x + 1];
        float a[4] = {0.f, 0.f, 0.f, 0.f};
        int64_t e = e0 + slot;
        for (; e + 12 < e1; e += 16) {
          int32_t u[4];
          float z[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) u[q] = er[e + 4 * q];
#pragma unroll
          for (int q = 0; q < 4; ++q) z[q] = Zr[static_cast<int64_t>(u[q]) * h + f];
#pragma unroll
          for (int q = 0; q < 4; ++q) a[q] += (u[q] < n_dst ? dinv[u[q]] : 1.0f) * z[q];
        }
        for (; e < e1; e += 4) {
          const int32_t u = er[e];
          a[0] += (u < n_dst ? dinv[u] : 1.0f) * Zr[static_cast<int64_t>(u) * h + f];
        }
        acc = (a[0] + a[1]) + (a[2] + a[3]);
      }
      acc += __shfl_xor(acc, 16);
      acc += __shfl_xor(acc, 32);
      if (x < n1 && slot == 0 && f < h) {
        const float dx = dinv[x];
        hv[wv * h + f] = fmaxf(dx * (acc + dx * Zr[x * h + f]) + (b1 ? b1[f] : 0.f), 0.f);
      }
      __syncthreads();
      chunk_logits(x0, nn);
      __syncthreads();
    }
  } else {
    for (int64_t x0 = 0; x0 < n1; x0 += nx) {
      const int64_t nn = n1 - x0 < nx ? n1 - x0 : nx;
      for (int64_t it = tid; it < nn * h; it += kEndsThreads) {
        const int64_t x = x0 + it / h;
        const int f = static_cast<int>(it % h);
        const int64_t e0 = dp[x], e1 = dp[x + 1];
        float acc = 0.f;
        // eight players' loads in flight at a time, summed in player order
        for (int64_t eb = e0; eb < e1; eb += 8) {
          int32_t u[8];
          float z[8];
#pragma unroll
          for (int q = 0; q < 8; ++q) u[q] = eb + q < e1 ? er[eb + q] : 0;
#pragma unroll
          for (int q = 0; q < 8; ++q) z[q] = eb + q < e1 ? Zr[static_cast<int64_t>(u[q]) * h + f] : 0.f;
#pragma unroll
          for (int q = 0; q < 8; ++q)
            if (eb + q < e1) acc += (u[q] < n_dst ? dinv[u[q]] : 1.0f) * z[q];
        }
        const float dx = dinv[x];
        hv[it] = fmaxf(dx * (acc + dx * Zr[x * h + f]) + (b1 ? b1[f] : 0.f), 0.f);
      }
      __syncthreads();
      chunk_logits(x0, nn);
      __syncthreads();
    }
  }
  for (int c = tid; c < C; c += kEndsThreads) {
    float t = 0.f;
    for (int f = 0; f < h; ++f) t += he[f] * w2[static_cast<int64_t>(f) * C + c];
    te[c] = t;
  }
  __syncthreads();
  // layer 2 at the target, one wavefront per class: lanes take the target's
  // players in turn (the source of player x - 1 is node x of H_1), summed by
  // a butterfly
  const int64_t indeg = dp[1];
  const float dv = dinv[0];
  for (int c = wv; c < C; c += kEndsThreads / 64) {
    float acc = 0.f;
    for (int64_t e = lane; e < indeg; e += 64) {
      const int32_t u = er[e];
      acc += dinv[u] * tt[static_cast<int64_t>(u) * C + c];
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
    if (lane == 0) {
      const float bias = b2 ? b2[c] : 0.f;
      sp_y[c] = d0 * (0.0f + d0 * te[c]) + bias;
      sp_y[C + c] = dv * (acc + dv * tt[c]) + bias;
    }
  }
  __syncthreads();
  if (tid == 0) pick_class(sp_y, C, requested, ctl, class_out, f_empty_full);
}

template <bool S>
__global__ void __launch_bounds__(kEndsThreads) k_eval_ends(const int32_t* __restrict__ dst_ptr,
                                                             const int32_t* __restrict__ edge_src, int64_t n_dst,
                                                             int64_t n1, int64_t M, float* Zc,
                                                             const float* __restrict__ XW1,
                                                             const int32_t* __restrict__ node_gid, int64_t n_nodes,
                                                             const float* __restrict__ b1,
                                                             const float* __restrict__ W2,
                                                             const float* __restrict__ b2, int h, int C,
                                                             float* __restrict__ sp_y, int requested, int32_t* ctl,
                                                             int32_t* class_out, float* f_empty_full) {
  ends_l2_body<S>(dst_ptr, edge_src, n_dst, n1, M, Zc, XW1, node_gid, n_nodes, b1, W2, b2, h, C, sp_y, requested,
                  ctl, class_out, f_empty_full);
}

// One launch of k_eval_ends for a single subgraph (staged when it fits).
void launch_ends(hipStream_t s, const gnnshap_subgraph* sg, int64_t n_dst, int64_t n1, int64_t n_nodes, float* Zc,
                 const float* XW1, const float* b1, const float* W2, const float* b2, int h, int C, float* sp_y,
                 int requested, int32_t* ctl, int32_t* class_out, float* f_empty_full) {
  bool S = false;
  const size_t lds = ends_launch_lds(n_dst, n1, n_nodes, sg->num_edges, h, C, &S);
  if (S)
    k_eval_ends<true><<<1, kEndsThreads, lds, s>>>(sg->dst_ptr, sg->edge_src, n_dst, n1, sg->num_edges, Zc, XW1,
                                                   sg->node_gid, n_nodes, b1, W2, b2, h, C, sp_y, requested, ctl,
                                                   class_out, f_empty_full);
  else
    k_eval_ends<false><<<1, kEndsThreads, lds, s>>>(sg->dst_ptr, sg->edge_src, n_dst, n1, sg->num_edges, Zc, XW1,
                                                    sg->node_gid, n_nodes, b1, W2, b2, h, C, sp_y, requested, ctl,
                                                    class_out, f_empty_full);
}

template <int FPT>
__global__ void __launch_bounds__(256) k_eval_l2(
    const uint64_t* __restrict__ masks, int64_t wpr, const int32_t* __restrict__ rows, int64_t row_off,
    int64_t cap, const int32_t* dyn_count, const int32_t* __restrict__ dst_ptr,
    const int32_t* __restrict__ edge_src, int64_t n_dst, int64_t n1, const float* __restrict__ Zc,
    const float* __restrict__ b1, const float* __restrict__ W2, const float* __restrict__ b2, int h, int C,
    const int32_t* __restrict__ ctl, bool all_classes, int tbr, float* __restrict__ y_rows,
    float* __restrict__ y_all) {
  eval_l2_body<FPT>(masks, wpr, rows, row_off, cap, dyn_count, dst_ptr, edge_src, n_dst, n1, Zc, b1, W2, b2, h, C,
                    ctl, all_classes, tbr, y_rows, y_all, blockIdx.x);
}

__global__ void k_pick_class(const float* __restrict__ sp_y, int C, int requested, int32_t* ctl,
                             int32_t* class_out, float* f_empty_full) {
  pick_class(sp_y, C, requested, ctl, class_out, f_empty_full);
}

// A coalition is evaluated only if it holds an in-edge of v (players [0, indeg v)).
__device__ __forceinline__ void live_rows_of(const uint64_t* __restrict__ masks, int64_t wpr, int64_t k,
                                             const int32_t* __restrict__ dst_ptr, int32_t* ctl,
                                             int32_t* live_rows, uint8_t* live_flag) {
  const int lane = threadIdx.x & 63;
  const int64_t indeg = dst_ptr[1];
  const int64_t nwords = (indeg + 63) >> 6;
  for (int64_t b0 = static_cast<int64_t>(blockIdx.x) * blockDim.x; b0 < k;
       b0 += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const int64_t b = b0 + threadIdx.x;
    bool live = false;
    if (b < k) {
      const uint64_t* mrow = masks + b * wpr;
      for (int64_t w = 0; w < nwords; ++w) {
        uint64_t word = mrow[w];
        const int64_t rem = indeg - w * 64;
        if (rem < 64) word &= (uint64_t(1) << rem) - 1;
        if (word) {
          live = true;
          break;
        }
      }
      live_flag[b] = live ? 1 : 0;
    }
    const uint64_t bal = __ballot(live);
    if (bal) {
      int base = 0;
      if (lane == 0) base = atomicAdd(&ctl[1], __popcll(bal));
      base = __shfl(base, 0);
      if (live) live_rows[base + __popcll(bal & ((1ull << lane) - 1ull))] = static_cast<int32_t>(b);
    }
  }
}

__global__ void __launch_bounds__(256) k_live(const uint64_t* __restrict__ masks, int64_t wpr,
                                              int64_t k, const int32_t* __restrict__ dst_ptr,
                                              int32_t* ctl, int32_t* live_rows, uint8_t* live_flag) {
  live_rows_of(masks, wpr, k, dst_ptr, ctl, live_rows, live_flag);
}

__global__ void k_fill_pruned(const uint8_t* __restrict__ live_flag, int64_t k,
                              const float* __restrict__ f_empty_full, float* __restrict__ y) {
  const float f0 = f_empty_full[0];
  for (int64_t b = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; b < k;
       b += static_cast<int64_t>(gridDim.x) * blockDim.x)
    if (!live_flag[b]) y[b] = f0;
}

typedef float f32x4_t __attribute__((ext_vector_type(4)));

// Z[r, :] = X[r, :] W for 16 rows per workgroup, h = 16 NT columns, fp32
// MFMA 16x16x4.  The KW wavefronts split K into KW parts and each lane
// group of 16 lanes takes a quarter of its wavefront's range, so every MFMA
// sums four k; the KW partial 16 x h tiles are added in LDS in a fixed order
// (no atomics: the result does not depend on scheduling).  Narrow outputs
// use 16 wavefronts: a 16-row tile then has four times as many loads in
// flight (the kernel is bound by their latency, not by the MFMAs).
template <int NT, int KW>
__global__ void __launch_bounds__(KW * 64) k_transform(const float* __restrict__ X, int64_t n, int d,
                                                       const float* __restrict__ W, int h, float* __restrict__ Z) {
  __shared__ float part[KW][16][16 * NT + 1];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane >> 4, c = lane & 15;
  const int64_t r0 = static_cast<int64_t>(blockIdx.x) * 16;
  const int64_t row = r0 + c;
  const int kq = (d + KW - 1) / KW;
  const int kb = wave * kq;
  const int ke = kb + kq < d ? kb + kq : d;
  const int kg = (kq + 3) / 4;
  const int k0 = kb + g * kg;
  f32x4_t acc[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) acc[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  const float* xr = X + (row < n ? row : 0) * static_cast<int64_t>(d);
  const int k1 = ke < k0 + kg ? ke : k0 + kg;     // this lane group's k range [k0, k1)
  // sixteen steps at a time: every load of a batch is issued before its products
  for (int s0 = 0; s0 < kg; s0 += 16) {
    float a[16], b[16][NT];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int k = k0 + s0 + i;
      const bool kin = k < k1;
      a[i] = (kin && row < n) ? xr[k] : 0.f;
#pragma unroll
      for (int t = 0; t < NT; ++t) b[i][t] = kin ? W[static_cast<int64_t>(k) * h + t * 16 + c] : 0.f;
    }
#pragma unroll
    for (int i = 0; i < 16; ++i)
#pragma unroll
      for (int t = 0; t < NT; ++t) acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[i][t], acc[t], 0, 0, 0);
  }
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int r = 0; r < 4; ++r) part[wave][4 * g + r][t * 16 + c] = acc[t][r];
  __syncthreads();
  for (int idx = threadIdx.x; idx < 16 * h; idx += KW * 64) {
    const int i = idx / h, j = idx % h;
    if (r0 + i < n) {
      float v = 0.f;
#pragma unroll
      for (int q = 0; q < KW; q += 4) v += (part[q][i][j] + part[q + 1][i][j]) + (part[q + 2][i][j] + part[q + 3][i][j]);
      Z[(r0 + i) * h + j] = v;
    }
  }
}

int launch_gemm(hipStream_t s, const float* A, int64_t lda, const int32_t* arow, const float* abias,
                const float* B, int64_t ldb, float* C, int64_t ldc, int64_t m0, int64_t rows, int64_t N,
                int64_t K, const int32_t* dyn = nullptr, int64_t dyn_off = 0, int64_t dyn_cap = 0,
                int64_t dyn_mult = 0) {
  if (rows <= 0) return GNNSHAP_OK;
  dim3 grid(static_cast<unsigned>(gnnshap::ceil_div(rows, 64)), static_cast<unsigned>(gnnshap::ceil_div(N, 64)));
  GS_TIMED("k_gemm", s);
  k_gemm<<<grid, 256, 0, s>>>(A, lda, arow, abias, B, ldb, C, ldc, m0, rows, N, K, dyn, dyn_off,
                              dyn_cap, dyn_mult);
  GS_LAUNCHED();
  return GNNSHAP_OK;
}

int launch_aggregate(hipStream_t s, int h, const uint64_t* masks, int64_t wpr, const int32_t* rows,
                     int64_t row_off, int64_t cap, const int32_t* dyn, const gnnshap_subgraph* sg,
                     const Shape& sh, const float* dinv, const float* Zc, const float* Zb,
                     int64_t nd_prev, const float* bias, float* Hout, int64_t nd_out) {
  int fpt = 16;
  while (fpt > 1 && 8 * (fpt / 2) >= h) fpt /= 2;
  const int fs = 8 * fpt;
  const int64_t n_tiles = gnnshap::ceil_div(cap, kTB);
  const int n_slices = static_cast<int>(gnnshap::ceil_div(h, fs));
  const int64_t blocks = n_tiles * nd_out * n_slices;
  if (blocks > INT32_MAX) return gnnshap::fail(GNNSHAP_EUNSUPPORTED, "aggregation grid too large");
  const unsigned g = static_cast<unsigned>(blocks);
  GS_TIMED("k_aggregate", s);
#define GS_AGG(F)                                                                                  \
  k_aggregate<F><<<g, 256, 0, s>>>(masks, wpr, rows, row_off, cap, dyn, sg->dst_ptr, sg->edge_src, \
                                   sh.n_dst, dinv, Zc, Zb, nd_prev, bias, Hout, nd_out, h, n_tiles, \
                                   n_slices)
  switch (fpt) {
    case 1: GS_AGG(1); break;
    case 2: GS_AGG(2); break;
    case 4: GS_AGG(4); break;
    case 8: GS_AGG(8); break;
    default: GS_AGG(16); break;
  }
#undef GS_AGG
  GS_LAUNCHED();
  return GNNSHAP_OK;
}

// Runs degrees -> layers 1..L-1 -> final for `cap` rows (or a device count).
size_t fused_lds_bytes(const Shape& sh, int64_t tbr, int ncls, int fs) {
  return sizeof(float) * (static_cast<size_t>(tbr) * sh.n_dst + static_cast<size_t>(tbr) * sh.nd[1] * ncls +
                          static_cast<size_t>(kChunkE) * fs) + sizeof(int32_t) * kChunkE;
}

int feature_split(int h) {
  int fpt = 16;
  while (fpt > 1 && 8 * (fpt / 2) >= h) fpt /= 2;
  return fpt;
}

// The fused two-layer kernel applies when its LDS fits; returns false otherwise.
bool fused_l2_ok(const Shape& sh, int64_t cap, bool all_classes) {
  if (sh.L != 2 || sh.hops < 2) return false;
  const int64_t tbr = cap < kTB ? cap : kTB;
  const int fs = 8 * feature_split(sh.dims[1]);
  return fused_lds_bytes(sh, tbr, all_classes ? sh.dims[2] : 1, fs) <= 65536;
}

// Whether the end coalitions take k_eval_ends (two-layer models, hops >= 2).
bool ends_ok(const Shape& sh) {
  return sh.L == 2 && sh.hops >= 2 && ends_lds_bytes(sh.n_dst, sh.nd[1], sh.dims[1], sh.dims[2]) <= 65536;
}

int launch_fused_l2(hipStream_t s, const gnnshap_subgraph* sg, const gnnshap_gcn* m, const Shape& sh, const Ws& w,
                    const uint64_t* masks, const int32_t* rows, int64_t row_off, int64_t cap, const int32_t* dyn,
                    bool all_classes, float* y_rows) {
  const int tbr = static_cast<int>(cap < kTB ? cap : kTB);
  const int h = sh.dims[1], C = sh.dims[2];
  const int fpt = feature_split(h);
  const size_t lds = fused_lds_bytes(sh, tbr, all_classes ? C : 1, 8 * fpt);
  const unsigned g = static_cast<unsigned>(gnnshap::ceil_div(cap, tbr));
  const float* b1 = m->b ? m->b[0] : nullptr;
  const float* b2 = m->b ? m->b[1] : nullptr;
#define GS_L2(F)                                                                                          \
  k_eval_l2<F><<<g, 256, lds, s>>>(masks, sh.wpr, rows, row_off, cap, dyn, sg->dst_ptr, sg->edge_src,      \
                                   sh.n_dst, sh.nd[1], w.Zc[1], b1, m->W[1], b2, h, C, w.ctl, all_classes, \
                                   tbr, y_rows, w.sp_y)
  GS_TIMED("k_eval_l2", s);
  const size_t lds_rows = rows_pass_lds(sh.n_dst, sh.nd[1], sg->num_edges, h);
  if (!all_classes && row_off == 0 && lds_rows > 0) {
    const unsigned gr = static_cast<unsigned>(gnnshap::ceil_div(cap, rows_pass_block(h)));
    if (h <= 16)
      k_eval_rows_mx<<<gr, kMxRows, lds_rows, s>>>(masks, sh.wpr, rows, cap, dyn, sg->dst_ptr, sg->edge_src, sh.n_dst,
                                                   sh.nd[1], sg->num_edges, w.Zc[1], nullptr, b1, m->W[1], b2, h, C,
                                                   w.ctl, nullptr, y_rows);
    else
      k_eval_rows<32><<<gr, kRowsPerBlock, lds_rows, s>>>(masks, sh.wpr, rows, cap, dyn, sg->dst_ptr, sg->edge_src,
                                                          sh.n_dst, sh.nd[1], sg->num_edges, w.Zc[1], nullptr, b1,
                                                          m->W[1], b2, h, C, w.ctl, nullptr, y_rows);
  } else {
    switch (fpt) {
      case 1: GS_L2(1); break;
      case 2: GS_L2(2); break;
      case 4: GS_L2(4); break;
      case 8: GS_L2(8); break;
      default: GS_L2(16); break;
    }
  }
#undef GS_L2
  GS_LAUNCHED();
  return GNNSHAP_OK;
}

int run_pass(hipStream_t s, const gnnshap_subgraph* sg, const gnnshap_gcn* m, const Shape& sh,
             const Ws& w, const uint64_t* masks, const int32_t* rows, int64_t row_off, int64_t cap,
             const int32_t* dyn, bool all_classes, float* y_rows) {
  if (fused_l2_ok(sh, cap, all_classes))
    return launch_fused_l2(s, sg, m, sh, w, masks, rows, row_off, cap, dyn, all_classes, y_rows);
  const int L = sh.L;
  k_degrees<<<gnnshap::grid_for(cap * sh.n_dst, 256), 256, 0, s>>>(masks, sh.wpr, rows, row_off, cap,
                                                                    dyn, sg->dst_ptr, sh.n_dst, w.dinv);
  GS_LAUNCHED();
  for (int j = 1; j < L; ++j) {
    const float* Zb = j >= 2 ? w.Zb[j] : nullptr;
    const float* bias = m->b ? m->b[j - 1] : nullptr;
    if (int st = launch_aggregate(s, sh.dims[j], masks, sh.wpr, rows, row_off, cap, dyn, sg, sh, w.dinv,
                                  w.Zc[j], Zb, sh.nd[j - 1], bias, w.Hb[j], sh.nd[j]))
      return st;
    if (j + 1 < L) {
      if (int st = launch_gemm(s, w.Hb[j], sh.dims[j], nullptr, nullptr, m->W[j], sh.dims[j + 1], w.Zb[j + 1],
                               sh.dims[j + 1], 0, cap * sh.nd[j], sh.dims[j + 1], sh.dims[j], dyn, row_off,
                               cap, sh.nd[j]))
        return st;
    }
  }
  const int C = sh.dims[L];
  const bool one = L == 1;
  const float* Hb = one ? nullptr : w.Hb[L - 1];
  const float* Hc = one ? w.Zc[1] : w.Bc[L - 1];
  const int64_t nd_last = one ? 0 : sh.nd[L - 1];
  const int h = one ? 1 : sh.dims[L - 1];
  k_final<<<static_cast<unsigned>(gnnshap::ceil_div(cap, 4)), 256, 0, s>>>(
      masks, sh.wpr, rows, row_off, cap, dyn, sg->dst_ptr, sg->edge_src, sh.n_dst, w.dinv, Hb, Hc,
      nd_last, h, m->W[L - 1], m->b ? m->b[L - 1] : nullptr, C, one, w.ctl, all_classes, y_rows, w.sp_y);
  GS_LAUNCHED();
  return GNNSHAP_OK;
}

// ---- multi-target path: one job per blockIdx.y -------------------------------------------

__global__ void k_init_batch(const gnnshap::EvalJob* __restrict__ jobs) {
  const gnnshap::EvalJob J = jobs[blockIdx.y];
  const int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (t < 8) J.ctl[t] = 0;
  if (t < 2) J.sp_rows[t] = static_cast<int32_t>(t);
  for (int64_t w = t; w < J.wpr; w += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    J.sp_masks[w] = 0;
    const int64_t lo = w * 64;
    const int64_t nb = J.M - lo >= 64 ? 64 : J.M - lo;
    J.sp_masks[J.wpr + w] = nb >= 64 ? ~uint64_t(0) : ((uint64_t(1) << nb) - 1);
  }
}

__global__ void k_gather_batch(const gnnshap::EvalJob* __restrict__ jobs, const float* __restrict__ XW1, int h) {
  const gnnshap::EvalJob J = jobs[blockIdx.y];
  const int64_t total = J.n_nodes * h;
  for (int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; t < total;
       t += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const int64_t u = t / h, f = t % h;
    J.Zc1[t] = XW1[static_cast<int64_t>(J.node_gid[u]) * h + f];
  }
}

// The end coalitions of every job.
template <bool S>
__global__ void __launch_bounds__(kEndsThreads) k_eval_ends_batch(const gnnshap::EvalJob* __restrict__ jobs,
                                                                   gnnshap::EvalModel md, bool gather) {
  const gnnshap::EvalJob J = jobs[blockIdx.x];
  ends_l2_body<S>(J.dst_ptr, J.edge_src, J.n_dst, J.n1, J.M, J.Zc1, gather ? md.XW1 : nullptr, J.node_gid,
                  J.n_nodes, md.b1, md.W2, md.b2, md.h, md.C, J.sp_y, md.target_class, J.ctl, J.cls_out, J.fef);
}

// Main pass of the jobs that do not take the one-thread-per-coalition kernel.
template <int FPT>
__global__ void __launch_bounds__(256) k_eval_l2_batch(const gnnshap::EvalJob* __restrict__ jobs,
                                                       gnnshap::EvalModel md, int tbr) {
  const gnnshap::EvalJob J = jobs[blockIdx.y];
  if (!J.rows_ok)
    eval_l2_body<FPT>(J.masks, J.wpr, J.live_rows, 0, J.k, J.ctl + 1, J.dst_ptr, J.edge_src, J.n_dst, J.n1, J.Zc1,
                      md.b1, md.W2, md.b2, md.h, md.C, J.ctl, false, tbr, J.y, J.sp_y, blockIdx.x);
}

// Main pass of the jobs that take the one-thread-per-coalition kernel;
// all: every row of the job (pruned rows get f(empty) on the way), else the
// live rows listed by k_live_batch.
__global__ void __launch_bounds__(kMxRows) k_eval_rows_mx_batch(const gnnshap::EvalJob* __restrict__ jobs,
                                                                gnnshap::EvalModel md, bool all) {
  const gnnshap::EvalJob J = jobs[blockIdx.y];
  if (!J.rows_ok) return;
  eval_rows_mx_body(J.masks, J.wpr, all ? nullptr : J.live_rows, J.k, all ? nullptr : J.ctl + 1, J.dst_ptr,
                    J.edge_src, J.n_dst, J.n1, J.M, J.Zc1, nullptr, md.b1, md.W2, md.b2, md.h, md.C, J.ctl, J.fef,
                    J.y, blockIdx.x);
}

template <int H>
__global__ void __launch_bounds__(kRowsPerBlock) k_eval_rows_batch(const gnnshap::EvalJob* __restrict__ jobs,
                                                                   gnnshap::EvalModel md, bool all) {
  const gnnshap::EvalJob J = jobs[blockIdx.y];
  if (!J.rows_ok) return;
  eval_rows_body<H>(J.masks, J.wpr, all ? nullptr : J.live_rows, J.k, all ? nullptr : J.ctl + 1, J.dst_ptr,
                    J.edge_src, J.n_dst, J.n1, J.M, J.Zc1, nullptr, md.b1, md.W2, md.b2, md.h, md.C, J.ctl, J.fef,
                    J.y, blockIdx.x);
}

__global__ void __launch_bounds__(256) k_live_batch(const gnnshap::EvalJob* __restrict__ jobs) {
  const gnnshap::EvalJob J = jobs[blockIdx.y];
  live_rows_of(J.masks, J.wpr, J.k, J.dst_ptr, J.ctl, J.live_rows, J.live_flag);
}

__global__ void k_fill_pruned_batch(const gnnshap::EvalJob* __restrict__ jobs) {
  const gnnshap::EvalJob J = jobs[blockIdx.y];
  const float f0 = J.fef[0];
  for (int64_t b = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; b < J.k;
       b += static_cast<int64_t>(gridDim.x) * blockDim.x)
    if (!J.live_flag[b]) J.y[b] = f0;
}

}  // namespace

extern "C" int gnnshap_eval_workspace(const gnnshap_subgraph* sg, const gnnshap_gcn* m, int64_t k,
                                      size_t* bytes) {
  gnnshap::clear_error();
  if (!bytes || k < 1) return gnnshap::fail(GNNSHAP_EINVAL, "bad arguments");
  Shape sh;
  if (int st = make_shape(sg, m, k, &sh)) return st;
  gnnshap::Carver c(nullptr);
  carve(c, sh);
  *bytes = c.bytes();
  return GNNSHAP_OK;
}

// gnnshap_eval_coalitions; pairs: rows b and b + k/2 are complements (the
// sampler's layout), which the wide path uses to contract half of the rows.
int gnnshap::eval_coalitions_impl(const gnnshap_subgraph* sg, const gnnshap_gcn* m, const float* X,
                                  int32_t target_class, const uint64_t* masks, int64_t k, int64_t words_per_row,
                                  float* y, float* f_empty_full, int32_t* class_out, void* ws, size_t ws_bytes,
                                  void* stream, bool pairs) {
  GS_TRY_BEGIN
  gnnshap::clear_error();
  if (k < 1) return gnnshap::fail(GNNSHAP_EINVAL, "k must be >= 1");
  Shape sh;
  if (int st = make_shape(sg, m, k, &sh)) return st;
  if ((!X && !m->XW1) || !masks || !y || !f_empty_full || !ws || !m->W)
    return gnnshap::fail(GNNSHAP_EINVAL, "null argument");
  for (int l = 0; l < sh.L; ++l)
    if (!m->W[l]) return gnnshap::fail(GNNSHAP_EINVAL, "null weight matrix %d", l);
  if (!sg->node_gid || !sg->dst_ptr || !sg->edge_src) return gnnshap::fail(GNNSHAP_EINVAL, "null subgraph arrays");
  if (words_per_row != sh.wpr) return gnnshap::fail(GNNSHAP_EINVAL, "words_per_row != ceil(M/64)");
  if (target_class >= sh.dims[sh.L] || target_class < -1) return gnnshap::fail(GNNSHAP_EINVAL, "target_class out of range");
  if (k > INT32_MAX) return gnnshap::fail(GNNSHAP_EINVAL, "k too large");
  gnnshap::Carver need(nullptr);
  carve(need, sh);
  if (ws_bytes < need.bytes()) return gnnshap::fail(GNNSHAP_ECAPACITY, "eval workspace needs %zu bytes", need.bytes());
  gnnshap::Carver cv(ws);
  const Ws w = carve(cv, sh);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int L = sh.L;

  // Two-layer models whose coalitions all fit the one-thread-per-coalition
  // kernel in one pass take two launches: the end coalitions (with the
  // class), then every row (pruned rows get f(empty) on the way), reading
  // X W_1 through the subgraph's node ids when it is given.
  const size_t lds_rows = rows_pass_lds(sh.n_dst, sh.nd[1], sg->num_edges, sh.dims[1]);
  const bool direct = ends_ok(sh) && fused_l2_ok(sh, k, false) && lds_rows > 0 && sh.tile >= k &&
                      gnnshap::ceil_div(k, kRowsPerBlock) <= INT32_MAX;
  if (direct) {
    if (!m->XW1) {
      if (int st = launch_gemm(s, X, sh.dims[0], sg->node_gid, nullptr, m->W[0], sh.dims[1], w.Zc[1], sh.dims[1], 0,
                               sh.n_nodes, sh.dims[1], sh.dims[0]))
        return st;
    }
    const float* Zsrc = w.Zc[1];
    const int32_t* zidx = nullptr;
    const float* b1 = m->b ? m->b[0] : nullptr;
    const float* b2 = m->b ? m->b[1] : nullptr;
    launch_ends(s, sg, sh.n_dst, sh.nd[1], sh.n_nodes, w.Zc[1], m->XW1, b1, m->W[1], b2, sh.dims[1], sh.dims[2],
                w.sp_y, target_class, w.ctl, class_out, f_empty_full);
    GS_LAUNCHED();
    const unsigned gr = static_cast<unsigned>(gnnshap::ceil_div(k, rows_pass_block(sh.dims[1])));
    GS_TIMED(sh.dims[1] <= 16 ? "k_eval_rows_mx" : "k_eval_rows", s);
    if (sh.dims[1] <= 16)
      k_eval_rows_mx<<<gr, kMxRows, lds_rows, s>>>(masks, sh.wpr, nullptr, k, nullptr, sg->dst_ptr, sg->edge_src,
                                                   sh.n_dst, sh.nd[1], sg->num_edges, Zsrc, zidx, b1, m->W[1], b2,
                                                   sh.dims[1], sh.dims[2], w.ctl, f_empty_full, y);
    else
      k_eval_rows<32><<<gr, kRowsPerBlock, lds_rows, s>>>(masks, sh.wpr, nullptr, k, nullptr, sg->dst_ptr,
                                                          sg->edge_src, sh.n_dst, sh.nd[1], sg->num_edges, Zsrc, zidx,
                                                          b1, m->W[1], b2, sh.dims[1], sh.dims[2], w.ctl,
                                                          f_empty_full, y);
    GS_LAUNCHED();
    return GNNSHAP_OK;
  }

  k_init<<<gnnshap::grid_for(sh.wpr, 256, 64), 256, 0, s>>>(w.ctl, w.sp_masks, w.sp_rows, sh.wpr, sg->num_edges);
  GS_LAUNCHED();
  // Constant rows: Z^1 = X[V_c] W_1 (gathered from X W_1 when given), then the boundary chain.
  if (m->XW1) {
    k_gather_rows<<<gnnshap::grid_for(sh.n_nodes * sh.dims[1], 256, 2048), 256, 0, s>>>(m->XW1, sg->node_gid,
                                                                                        sh.n_nodes, sh.dims[1], w.Zc[1]);
    GS_LAUNCHED();
  } else if (int st = launch_gemm(s, X, sh.dims[0], sg->node_gid, nullptr, m->W[0], sh.dims[1], w.Zc[1], sh.dims[1],
                                  0, sh.n_nodes, sh.dims[1], sh.dims[0])) {
    return st;
  }
  for (int j = 1; j < L; ++j) {
    if (!sh.bnd[j]) continue;
    k_bias_relu<<<gnnshap::grid_for((sh.bnd1 - sh.bnd0) * sh.dims[j], 256, 1024), 256, 0, s>>>(
        w.Zc[j], m->b ? m->b[j - 1] : nullptr, w.Bc[j], sh.bnd0, sh.bnd1, sh.dims[j]);
    GS_LAUNCHED();
    if (j + 1 < L) {
      if (int st = launch_gemm(s, w.Bc[j], sh.dims[j], nullptr, nullptr, m->W[j], sh.dims[j + 1], w.Zc[j + 1],
                               sh.dims[j + 1], sh.bnd0, sh.bnd1 - sh.bnd0, sh.dims[j + 1], sh.dims[j]))
        return st;
    }
  }
  // f(empty) and f(E_c) for every class, then the explained class.
  if (sh.wide && L == 2) {
    const float* b1 = m->b ? m->b[0] : nullptr;
    const float* b2 = m->b ? m->b[1] : nullptr;
    if (int st = gnnshap::launch_wide_ends(sh.ws, w.wide, sg, w.Zc[1], b1, m->W[1], b2, target_class, w.sp_y, w.ctl,
                                           class_out, f_empty_full, s))
      return st;
    return gnnshap::launch_wide(sh.ws, w.wide, sg, masks, sh.wpr, w.Zc[1], b1, m->W[1], b2, w.ctl, f_empty_full,
                                pairs, y, s);
  }
  if (sh.wide) {
    // three layers.  The end coalitions: layer 1, its transform by W_2, then
    // layer 2 and the output layer for every class
    const gnnshap::WideShape& ws = sh.ws;
    if (int st = gnnshap::launch_wide3_ends_l1(ws, w.wide, sg, w.Zc[1], m->b ? m->b[0] : nullptr, s)) return st;
    if (int st = launch_gemm(s, w.wide.hf, ws.h, nullptr, nullptr, m->W[1], ws.h2, w.wide.z2e, ws.h2, 0, ws.n1 + 1,
                             ws.h2, ws.h))
      return st;
    if (int st = gnnshap::launch_wide3_ends_l2(ws, w.wide, sg, w.Zc[2], m->b ? m->b[1] : nullptr, m->W[2],
                                               m->b ? m->b[2] : nullptr, target_class, w.sp_y, w.ctl, class_out,
                                               f_empty_full, s))
      return st;
    // every row: layer 1 and layer 2 at H_1 as contractions, the dense
    // transform by W_2 between them, in passes over the rows
    if (int st = gnnshap::launch_wide3_prep(ws, w.wide, sg, masks, sh.wpr, w.Zc[1], w.Zc[2], pairs, s)) return st;
    const int64_t nrows = pairs ? k / 2 : k;
    for (int64_t r0 = 0; r0 < nrows; r0 += ws.pass) {
      const int64_t nloc = std::min(ws.pass, nrows - r0);
      if (int st = gnnshap::launch_wide3_l1(ws, w.wide, sg, masks, sh.wpr, r0, nloc, w.Zc[1], m->b ? m->b[0] : nullptr,
                                            pairs, s))
        return st;
      if (ws.agg3) {
        // three hops: layer 2's sums at the target and its in-neighbours, then W_2 there only
        if (int st = gnnshap::launch_wide3_agg(ws, w.wide, sg, masks, sh.wpr, r0, nloc, pairs, s)) return st;
        if (int st = launch_gemm(s, w.wide.A3, ws.h, nullptr, nullptr, m->W[1], ws.h2, w.wide.Z2, ws.h2, 0,
                                 (pairs ? 2 : 1) * nloc * ws.n2, ws.h2, ws.h))
          return st;
        if (int st = gnnshap::launch_wide3_t(ws, w.wide, sg, masks, sh.wpr, r0, nloc, m->b ? m->b[1] : nullptr,
                                             m->W[2], w.ctl, pairs, s))
          return st;
        continue;
      }
      if (int st = launch_gemm(s, w.wide.H1, ws.h, nullptr, nullptr, m->W[1], ws.h2, w.wide.Z2, ws.h2, 0,
                               (pairs ? 2 : 1) * nloc * ws.n1, ws.h2, ws.h))
        return st;
      if (int st = gnnshap::launch_wide3_l2(ws, w.wide, sg, masks, sh.wpr, r0, nloc, m->b ? m->b[1] : nullptr,
                                            m->W[2], w.ctl, pairs, s))
        return st;
    }
    return gnnshap::launch_wide3_out(ws, w.wide, sg, masks, sh.wpr, m->b ? m->b[2] : nullptr, w.ctl, f_empty_full,
                                     pairs, y, s);
  }
  if (ends_ok(sh)) {
    launch_ends(s, sg, sh.n_dst, sh.nd[1], sh.n_nodes, w.Zc[1], nullptr, m->b ? m->b[0] : nullptr, m->W[1],
                m->b ? m->b[1] : nullptr, sh.dims[1], sh.dims[2], w.sp_y, target_class, w.ctl, class_out,
                f_empty_full);
    GS_LAUNCHED();
  } else {
    if (int st = run_pass(s, sg, m, sh, w, w.sp_masks, w.sp_rows, 0, 2, nullptr, true, nullptr)) return st;
    k_pick_class<<<1, 1, 0, s>>>(w.sp_y, sh.dims[L], target_class, w.ctl, class_out, f_empty_full);
    GS_LAUNCHED();
  }
  // Prediction pruning, then the live coalitions in passes of sh.tile rows.
  k_live<<<gnnshap::grid_for(k, 256, 4096), 256, 0, s>>>(masks, sh.wpr, k, sg->dst_ptr, w.ctl, w.live_rows,
                                                         w.live_flag);
  GS_LAUNCHED();
  for (int64_t off = 0; off < k; off += sh.tile) {
    const int64_t cap = std::min(sh.tile, k - off);
    if (int st = run_pass(s, sg, m, sh, w, masks, w.live_rows, off, cap, w.ctl + 1, false, y)) return st;
  }
  k_fill_pruned<<<gnnshap::grid_for(k, 256, 4096), 256, 0, s>>>(w.live_flag, k, f_empty_full, y);
  GS_LAUNCHED();
  return GNNSHAP_OK;
  GS_TRY_END
}

extern "C" int gnnshap_eval_coalitions(const gnnshap_subgraph* sg, const gnnshap_gcn* m, const float* X,
                                       int32_t target_class, const uint64_t* masks, int64_t k,
                                       int64_t words_per_row, float* y, float* f_empty_full,
                                       int32_t* class_out, void* ws, size_t ws_bytes, void* stream) {
  return gnnshap::eval_coalitions_impl(sg, m, X, target_class, masks, k, words_per_row, y, f_empty_full, class_out,
                                       ws, ws_bytes, stream, false);
}

extern "C" int gnnshap_eval_sampled_coalitions(const gnnshap_subgraph* sg, const gnnshap_gcn* m, const float* X,
                                               int32_t target_class, const uint64_t* masks, int64_t k,
                                               int64_t words_per_row, float* y, float* f_empty_full,
                                               int32_t* class_out, void* ws, size_t ws_bytes, void* stream) {
  if (k % 2) return gnnshap::fail(GNNSHAP_EINVAL, "sampled coalitions come in complement pairs: k must be even");
  return gnnshap::eval_coalitions_impl(sg, m, X, target_class, masks, k, words_per_row, y, f_empty_full, class_out,
                                       ws, ws_bytes, stream, true);
}

extern "C" int gnnshap_transform_features(const float* X, int64_t n, int32_t d, const float* W, int32_t h, float* Z,
                                          void* stream) {
  GS_TRY_BEGIN
  gnnshap::clear_error();
  if (!X || !W || !Z) return gnnshap::fail(GNNSHAP_EINVAL, "null argument");
  if (n < 1 || d < 1 || h < 1) return gnnshap::fail(GNNSHAP_EINVAL, "bad sizes");
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (h % 16 == 0 && h <= 128 && gnnshap::ceil_div(n, 16) <= INT32_MAX) {
    const unsigned g = static_cast<unsigned>(gnnshap::ceil_div(n, 16));
    GS_TIMED("k_transform", s);
    switch (h / 16) {
      case 1: k_transform<1, 16><<<g, 1024, 0, s>>>(X, n, d, W, h, Z); break;
      case 2: k_transform<2, 16><<<g, 1024, 0, s>>>(X, n, d, W, h, Z); break;
      case 3: k_transform<3, 4><<<g, 256, 0, s>>>(X, n, d, W, h, Z); break;
      case 4: k_transform<4, 4><<<g, 256, 0, s>>>(X, n, d, W, h, Z); break;
      case 5: k_transform<5, 4><<<g, 256, 0, s>>>(X, n, d, W, h, Z); break;
      case 6: k_transform<6, 4><<<g, 256, 0, s>>>(X, n, d, W, h, Z); break;
      case 7: k_transform<7, 4><<<g, 256, 0, s>>>(X, n, d, W, h, Z); break;
      default: k_transform<8, 4><<<g, 256, 0, s>>>(X, n, d, W, h, Z); break;
    }
    GS_LAUNCHED();
    return GNNSHAP_OK;
  }
  if (gnnshap::ceil_div(n, 64) > INT32_MAX || gnnshap::ceil_div(h, 64) > 65535)
    return gnnshap::fail(GNNSHAP_EUNSUPPORTED, "matrix too large");
  return launch_gemm(s, X, d, nullptr, nullptr, W, h, Z, h, 0, n, h, d);
  GS_TRY_END
}

// ---- multi-target path: host side --------------------------------------------------------

bool gnnshap::eval_batchable(const gnnshap_subgraph* sg, const gnnshap_gcn* m, int64_t k) {
  Shape sh;
  if (make_shape(sg, m, k, &sh) != GNNSHAP_OK) {
    clear_error();
    return false;
  }
  return m->XW1 && m->W && m->W[1] && sh.L == 2 && sh.hops >= 2 && sh.tile >= k && k <= INT32_MAX &&
         ends_ok(sh) && fused_l2_ok(sh, k, false);
}

size_t gnnshap::eval_slice_bytes(const gnnshap_subgraph* sg, const gnnshap_gcn* m, int64_t k) {
  Shape sh;
  if (make_shape(sg, m, k, &sh) != GNNSHAP_OK) return 0;
  Carver c(nullptr);
  carve(c, sh);
  return c.bytes();
}

void gnnshap::eval_carve_slice(void* base, const gnnshap_subgraph* sg, const gnnshap_gcn* m, int64_t k,
                               EvalJob* job) {
  Shape sh;
  make_shape(sg, m, k, &sh);
  Carver c(base);
  const Ws w = carve(c, sh);
  job->ctl = w.ctl;
  job->sp_masks = w.sp_masks;
  job->sp_rows = w.sp_rows;
  job->sp_y = w.sp_y;
  job->live_rows = w.live_rows;
  job->live_flag = w.live_flag;
  job->Zc1 = w.Zc[1];
}

int gnnshap::launch_eval_batch(const EvalJob* jobs, int64_t n, const EvalModel& md, int64_t max_nodes,
                               int64_t max_ndst, int64_t max_n1, int64_t max_wpr, int64_t max_k, int64_t rows_jobs,
                               size_t rows_lds, hipStream_t s) {
  if (n < 1) return GNNSHAP_OK;
  if (n > 65535) return fail(GNNSHAP_EUNSUPPORTED, "at most 65535 targets per batch");
  Shape sh;                          // the largest shapes of the batch, for LDS sizing
  sh.n_dst = max_ndst;
  sh.nd[1] = max_n1;
  const int fpt = feature_split(md.h);
  const int tb_main = static_cast<int>(max_k < kTB ? max_k : kTB);
  const size_t lds_ends = ends_lds_bytes(max_ndst, max_n1, md.h, md.C);
  const size_t lds_main = fused_lds_bytes(sh, tb_main, 1, 8 * fpt);
  if (lds_ends > 65536 || lds_main > 65536)
    return fail(GNNSHAP_EUNSUPPORTED, "batched evaluation needs %zu bytes of LDS", std::max(lds_ends, lds_main));
  const unsigned nn = static_cast<unsigned>(n);
  const bool all = rows_jobs == n;   // every job takes the one-thread-per-coalition kernel: two launches
  if (!all) {
    k_init_batch<<<dim3(grid_for(max_wpr, 256, 64), nn), 256, 0, s>>>(jobs);
    GS_LAUNCHED();
    k_gather_batch<<<dim3(grid_for(max_nodes * md.h, 256, 2048), nn), 256, 0, s>>>(jobs, md.XW1, md.h);
    GS_LAUNCHED();
  }
  {
    GS_TIMED("k_eval_ends_batch", s);
    bool S = false;
    const size_t lds = ends_launch_lds(max_ndst, max_n1, max_nodes, 64 * max_wpr, md.h, md.C, &S);
    if (S) k_eval_ends_batch<true><<<nn, kEndsThreads, lds, s>>>(jobs, md, all);
    else k_eval_ends_batch<false><<<nn, kEndsThreads, lds, s>>>(jobs, md, all);
  }
  GS_LAUNCHED();
  if (!all) {
    k_live_batch<<<dim3(grid_for(max_k, 256, 4096), nn), 256, 0, s>>>(jobs);
    GS_LAUNCHED();
#define GS_L2B(F, GRID, LDS, TBR) k_eval_l2_batch<F><<<GRID, 256, LDS, s>>>(jobs, md, TBR)
    GS_TIMED("k_eval_l2_batch", s);
    const dim3 g(static_cast<unsigned>(ceil_div(max_k, tb_main)), nn);
    switch (fpt) {
      case 1: GS_L2B(1, g, lds_main, tb_main); break;
      case 2: GS_L2B(2, g, lds_main, tb_main); break;
      case 4: GS_L2B(4, g, lds_main, tb_main); break;
      case 8: GS_L2B(8, g, lds_main, tb_main); break;
      default: GS_L2B(16, g, lds_main, tb_main); break;
    }
#undef GS_L2B
    GS_LAUNCHED();
  }
  if (rows_jobs > 0) {
    GS_TIMED(md.h <= 16 ? "k_eval_rows_mx_batch" : "k_eval_rows_batch", s);
    const dim3 g(static_cast<unsigned>(ceil_div(max_k, rows_pass_block(md.h))), nn);
    if (md.h <= 16) k_eval_rows_mx_batch<<<g, kMxRows, rows_lds, s>>>(jobs, md, all);
    else k_eval_rows_batch<32><<<g, kRowsPerBlock, rows_lds, s>>>(jobs, md, all);
  }
  GS_LAUNCHED();
  if (!all) {
    k_fill_pruned_batch<<<dim3(grid_for(max_k, 256, 4096), nn), 256, 0, s>>>(jobs);
    GS_LAUNCHED();
  }
  return GNNSHAP_OK;
}

// Whether a target's main pass takes the one-thread-per-coalition kernel, and its LDS.
size_t gnnshap::eval_rows_lds(const gnnshap_subgraph* sg, const gnnshap_gcn* m) {
  if (m->num_layers != 2) return 0;
  return rows_pass_lds(sg->num_dst, sg->hop_ptr[2], sg->num_edges, m->dims[1]);
}
