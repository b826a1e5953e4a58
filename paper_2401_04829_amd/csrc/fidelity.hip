// Fidelity of an explanation (eq. 7-8, Sec. 4.3; protocol of Sec. 4.6).
//
// Importance of a player is |phi| (Sec. 2.3), larger first, equal values by
// lower player index.  G_S keeps all players but the floor(s M) least
// important, G_{C \ S} all but the min(k, M) most important; both are
// evaluated as two deterministic coalitions by the coalition kernels, and a
// target's terms are |f(G_C) - f(G_S)| and |f(G_C) - f(G_{C\S})| for the
// explained output.
//
// The two player sets come from one workgroup per target: the n-th largest
// key (the float bits of |phi|, which order like the values) by a binary
// search over its 32 bits, each step a count over the players; then one pass
// in player order that ranks the players equal to that key by a prefix count
// (wave ballots) and writes the mask words with ballots.
#include <cmath>

#include "common.h"

namespace {

constexpr int kFidThreads = 1024;
constexpr int kFidWaves = kFidThreads / 64;

__device__ __forceinline__ uint32_t key_of(const float* __restrict__ phi, int64_t j) {
  return __float_as_uint(phi[j]) & 0x7FFFFFFFu;   // |phi| as ordered bits
}

// Number of players with key >= t (every thread gets it).
__device__ uint32_t count_ge(const float* __restrict__ phi, int64_t M, uint32_t t, uint32_t* red) {
  uint32_t c = 0;
  for (int64_t j = threadIdx.x; j < M; j += kFidThreads) c += key_of(phi, j) >= t ? 1u : 0u;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) c += __shfl_xor(c, off);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = c;
  __syncthreads();
  uint32_t s = 0;
  for (int i = 0; i < kFidWaves; ++i) s += red[i];
  return s;
}

// Row `row` of masks: bit j set iff player j is among the n most important
// (complemented within the M players when `complement`).
__device__ void write_top(const float* __restrict__ phi, int64_t M, int64_t n, bool complement, int64_t wpr,
                          uint64_t* __restrict__ out, uint32_t* red) {
  uint32_t thr = 0, need = 0;   // members: key > thr, and the first `need` players with key == thr
  bool all = n >= M, none = n <= 0;
  if (!all && !none) {
    // largest t with count(key >= t) >= n
    uint32_t lo = 0, hi = 0x7FFFFFFFu;
    while (lo < hi) {
      const uint32_t mid = lo + (hi - lo + 1) / 2;
      if (count_ge(phi, M, mid, red) >= static_cast<uint32_t>(n)) lo = mid; else hi = mid - 1;
    }
    thr = lo;
    const uint32_t above = thr == 0x7FFFFFFFu ? 0u : count_ge(phi, M, thr + 1, red);
    need = static_cast<uint32_t>(n) - above;
  }
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  uint32_t carry = 0;
  for (int64_t base = 0; base < M; base += kFidThreads) {
    const int64_t j = base + threadIdx.x;
    const bool valid = j < M;
    const uint32_t k = valid ? key_of(phi, j) : 0u;
    const bool eq = valid && !all && !none && k == thr;
    const bool gt = valid && !all && !none && k > thr;
    const uint64_t eqb = __ballot(eq);
    const uint32_t before = __popcll(eqb & ((1ull << lane) - 1ull));
    __syncthreads();
    if (lane == 0) red[wv] = __popcll(eqb);
    __syncthreads();
    uint32_t wave_off = 0, total = 0;
    for (int i = 0; i < kFidWaves; ++i) {
      if (i < wv) wave_off += red[i];
      total += red[i];
    }
    const bool in = all ? valid : (gt || (eq && carry + wave_off + before < need));
    const bool bit = valid && (complement ? !in : in);
    const uint64_t word = __ballot(bit);
    const int64_t w = (base >> 6) + wv;
    if (lane == 0 && w < wpr) out[w] = word;
    carry += total;
  }
}

__global__ void __launch_bounds__(kFidThreads) k_fid_masks(const float* __restrict__ phi, int64_t M, int64_t n_keep,
                                                          int64_t n_top, int64_t wpr, uint64_t* __restrict__ masks) {
  __shared__ uint32_t red[kFidWaves];
  write_top(phi, M, n_keep, false, wpr, masks, red);        // G_S
  write_top(phi, M, n_top, true, wpr, masks + wpr, red);    // G_{C \ S}
}

// out[0] = |f(G_C) - f(G_S)|, out[1] = |f(G_C) - f(G_{C\S})|, out[2] = f(G_C).
__global__ void k_fid_terms(const float* __restrict__ y, const float* __restrict__ fef, float* __restrict__ out) {
  if (threadIdx.x == 0) {
    const double full = fef[1];
    out[0] = static_cast<float>(fabs(full - static_cast<double>(y[0])));
    out[1] = static_cast<float>(fabs(full - static_cast<double>(y[1])));
    out[2] = fef[1];
  }
}

// avg[c] = mean over t of terms[t * stride + c], c = 0, 1 (fp64 sums in a fixed order).
__global__ void __launch_bounds__(256) k_fid_average(const float* __restrict__ terms, int64_t n, int64_t stride,
                                                     float* __restrict__ avg) {
  __shared__ double red[2][4];
  double s0 = 0.0, s1 = 0.0;
  for (int64_t t = threadIdx.x; t < n; t += 256) {
    s0 += terms[t * stride];
    s1 += terms[t * stride + 1];
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    s0 += __shfl_xor(s0, off);
    s1 += __shfl_xor(s1, off);
  }
  if ((threadIdx.x & 63) == 0) {
    red[0][threadIdx.x >> 6] = s0;
    red[1][threadIdx.x >> 6] = s1;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    const double a = (red[0][0] + red[0][1]) + (red[0][2] + red[0][3]);
    const double b = (red[1][0] + red[1][1]) + (red[1][2] + red[1][3]);
    avg[0] = static_cast<float>(a / static_cast<double>(n));
    avg[1] = static_cast<float>(b / static_cast<double>(n));
  }
}

struct FidWs {
  uint64_t* masks;
  float* y;
  float* fef;
  void* eval;
  size_t eval_bytes;
};

int fid_carve(const gnnshap_subgraph* sg, const gnnshap_gcn* m, void* base, FidWs* w, size_t* bytes) {
  size_t eb = 0;
  if (int st = gnnshap_eval_workspace(sg, m, 2, &eb)) return st;
  gnnshap::Carver c(base);
  const int64_t wpr = gnnshap::ceil_div(sg->num_edges, 64);
  w->masks = c.take<uint64_t>(2 * wpr);
  w->y = c.take<float>(2);
  w->fef = c.take<float>(2);
  w->eval = c.take<char>(eb);
  w->eval_bytes = eb;
  *bytes = c.bytes();
  return GNNSHAP_OK;
}

}  // namespace

extern "C" int gnnshap_fidelity_workspace(const gnnshap_subgraph* sg, const gnnshap_gcn* m, size_t* bytes) {
  gnnshap::clear_error();
  if (!sg || !m || !bytes) return gnnshap::fail(GNNSHAP_EINVAL, "null argument");
  if (sg->num_edges < 1) return gnnshap::fail(GNNSHAP_EINVAL, "the subgraph has no players");
  FidWs w;
  return fid_carve(sg, m, nullptr, &w, bytes);
}

extern "C" int gnnshap_fidelity(const gnnshap_subgraph* sg, const gnnshap_gcn* m, const float* X,
                                int32_t target_class, const float* phi, double sparsity, int64_t top_k, float* out,
                                void* ws, size_t ws_bytes, void* stream) {
  GS_TRY_BEGIN
  gnnshap::clear_error();
  if (!sg || !m || !X || !phi || !out || !ws) return gnnshap::fail(GNNSHAP_EINVAL, "null argument");
  if (sg->num_edges < 1) return gnnshap::fail(GNNSHAP_EINVAL, "the subgraph has no players");
  if (!(sparsity >= 0.0 && sparsity <= 1.0)) return gnnshap::fail(GNNSHAP_EINVAL, "sparsity must be in [0, 1]");
  if (top_k < 0) return gnnshap::fail(GNNSHAP_EINVAL, "top_k must be >= 0");
  FidWs w;
  size_t need = 0;
  if (int st = fid_carve(sg, m, nullptr, &w, &need)) return st;
  if (ws_bytes < need) return gnnshap::fail(GNNSHAP_ECAPACITY, "fidelity workspace needs %zu bytes", need);
  if (int st = fid_carve(sg, m, ws, &w, &need)) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t M = sg->num_edges;
  const int64_t wpr = gnnshap::ceil_div(M, 64);
  if (int st = gnnshap_fidelity_masks(phi, M, sparsity, top_k, w.masks, stream)) return st;
  if (int st = gnnshap_eval_coalitions(sg, m, X, target_class, w.masks, 2, wpr, w.y, w.fef, nullptr, w.eval,
                                       w.eval_bytes, stream))
    return st;
  k_fid_terms<<<1, 64, 0, s>>>(w.y, w.fef, out);
  GS_LAUNCHED();
  return GNNSHAP_OK;
  GS_TRY_END
}

extern "C" int gnnshap_fidelity_masks(const float* phi, int64_t M, double sparsity, int64_t top_k, uint64_t* masks,
                                      void* stream) {
  GS_TRY_BEGIN
  gnnshap::clear_error();
  if (!phi || !masks) return gnnshap::fail(GNNSHAP_EINVAL, "null argument");
  if (M < 1) return gnnshap::fail(GNNSHAP_EINVAL, "M must be >= 1");
  if (!(sparsity >= 0.0 && sparsity <= 1.0)) return gnnshap::fail(GNNSHAP_EINVAL, "sparsity must be in [0, 1]");
  if (top_k < 0) return gnnshap::fail(GNNSHAP_EINVAL, "top_k must be >= 0");
  const int64_t wpr = gnnshap::ceil_div(M, 64);
  const int64_t n_drop = static_cast<int64_t>(std::floor(sparsity * static_cast<double>(M)));
  const int64_t n_keep = M - (n_drop < M ? n_drop : M);
  const int64_t n_top = top_k < M ? top_k : M;
  {
    GS_TIMED("k_fid_masks", static_cast<hipStream_t>(stream));
    k_fid_masks<<<1, kFidThreads, 0, static_cast<hipStream_t>(stream)>>>(phi, M, n_keep, n_top, wpr, masks);
  }
  GS_LAUNCHED();
  return GNNSHAP_OK;
  GS_TRY_END
}

extern "C" int gnnshap_fidelity_average(const float* terms, int64_t n, int64_t stride, float* avg, void* stream) {
  GS_TRY_BEGIN
  gnnshap::clear_error();
  if (!terms || !avg) return gnnshap::fail(GNNSHAP_EINVAL, "null argument");
  if (n < 1 || stride < 2) return gnnshap::fail(GNNSHAP_EINVAL, "need n >= 1 targets and stride >= 2");
  k_fid_average<<<1, 256, 0, static_cast<hipStream_t>(stream)>>>(terms, n, stride, avg);
  GS_LAUNCHED();
  return GNNSHAP_OK;
  GS_TRY_END
}
