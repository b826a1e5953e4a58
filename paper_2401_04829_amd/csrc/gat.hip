// Coalition values of a two-layer graph attention network (App. E of the
// GNNShap paper: the explainer treats the model as a black box and is shown
// on a GAT with 8 heads).
//
// A coalition keeps its edges and every self loop.  Layer 1 (H heads of
// width F, concatenated, then ELU) at node x of H_1 under coalition S:
//     out1_h[x] = sum_{u in N_S(x) + x} a_h(u -> x) z_h[u] / sum a_h(u -> x)
// with z = X W_1 and a_h(u -> x) = exp(LeakyReLU(s_h[u] + d_h[x]) - m_h[x]),
// s_h = a_src,h . z_h, d_h = a_dst,h . z_h.  The logits, and therefore the
// unnormalised weights a_h, do not depend on the coalition: they are
// computed once per target (m_h[x] is the largest logit among all of x's
// candidate edges, so every weight is at most 1); a coalition only decides
// which of them enter the sums, i.e. the softmax is renormalised over the
// present edges.  Layer 2 (one head of width C) is needed at the target v
// only, and only through the class explained: with u2_src = W_2 a_src,2 and
// u2_dst = W_2 a_dst,2, the layer-2 logit of edge x -> v is
// LeakyReLU(out1[x] . u2_src + out1[v] . u2_dst) and the class value of x is
// out1[x] . W_2[:, c]; their softmax is accumulated online (running maximum).
// Layer 1 is computed only at v and at the in-neighbours of v whose edge to
// v is present (the others do not reach v).  A coalition without an in-edge
// of v has the value f(empty) (Sec. 3.4.1 holds for any message-passing
// model).
#include <algorithm>
#include <cmath>

#include "common.h"

namespace {

constexpr int kGatMaxFeat = 256;              // heads * head_dim
constexpr int kGatSlots = kGatMaxFeat / 64;   // features per lane
constexpr int kRowsWaves = 4;                 // coalitions per workgroup of the per-coalition kernel

struct GatDev {
  // subgraph
  const int32_t* gid;
  const int32_t* dst_ptr;
  const int32_t* esrc;
  int64_t n_nodes, n1, M, indeg_v;
  // model
  int32_t H, F, nf, C;
  const float* XW1;
  const float* att_src1;
  const float* att_dst1;
  const float* b1;
  const float* W2;
  const float* att_src2;
  const float* att_dst2;
  const float* b2;
  float slope;
  // workspace
  float* z1;     // n_nodes x nf
  float* ss1;    // n_nodes x H
  float* sd1;    // n1 x H
  float* w;      // M x H
  float* wself;  // n1 x H
  float* u2s;    // nf
  float* u2d;    // nf
  int32_t* cls;  // explained class
};

__device__ __forceinline__ float leaky(float x, float slope) { return x > 0.f ? x : slope * x; }
__device__ __forceinline__ float elu(float x) { return x > 0.f ? x : expm1f(x); }

__device__ __forceinline__ float wave_sum_f(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  return v;
}

// z1 rows of the subgraph's nodes and the per-head attention terms s (every
// node) and d (nodes of H_1).  Grid-stride over (node, feature) and (node, head).
__global__ void __launch_bounds__(256) k_gat_gather(GatDev g) {
  const int64_t tid = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (int64_t i = tid; i < g.n_nodes * g.nf; i += stride) {
    const int64_t u = i / g.nf, f = i % g.nf;
    g.z1[i] = g.XW1[static_cast<int64_t>(g.gid[u]) * g.nf + f];
  }
  for (int64_t i = tid; i < g.n_nodes * g.H; i += stride) {
    const int64_t u = i / g.H, h = i % g.H;
    const float* z = g.XW1 + static_cast<int64_t>(g.gid[u]) * g.nf + h * g.F;
    float s = 0.f, d = 0.f;
    for (int f = 0; f < g.F; ++f) {
      s += g.att_src1[h * g.F + f] * z[f];
      d += g.att_dst1[h * g.F + f] * z[f];
    }
    g.ss1[i] = s;
    if (u < g.n1) g.sd1[i] = d;
  }
}

// Unnormalised layer-1 weights of every candidate edge (players into H_1 and
// the self loops), shifted by each destination's largest logit; the layer-2
// attention vectors folded through W_2.
__global__ void __launch_bounds__(256) k_gat_weights(GatDev g) {
  const int64_t tid = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (int64_t i = tid; i < g.n1 * g.H; i += stride) {
    const int64_t x = i / g.H, h = i % g.H;
    const float d = g.sd1[i];
    const float lself = leaky(g.ss1[x * g.H + h] + d, g.slope);
    float m = lself;
    for (int32_t p = g.dst_ptr[x]; p < g.dst_ptr[x + 1]; ++p)
      m = fmaxf(m, leaky(g.ss1[static_cast<int64_t>(g.esrc[p]) * g.H + h] + d, g.slope));
    for (int32_t p = g.dst_ptr[x]; p < g.dst_ptr[x + 1]; ++p)
      g.w[static_cast<int64_t>(p) * g.H + h] = expf(leaky(g.ss1[static_cast<int64_t>(g.esrc[p]) * g.H + h] + d, g.slope) - m);
    g.wself[i] = expf(lself - m);
  }
  for (int64_t f = tid; f < g.nf; f += stride) {
    float s = 0.f, d = 0.f;
    for (int c = 0; c < g.C; ++c) {
      s += g.W2[f * g.C + c] * g.att_src2[c];
      d += g.W2[f * g.C + c] * g.att_dst2[c];
    }
    g.u2s[f] = s;
    g.u2d[f] = d;
  }
}

// Layer-1 output of node x for this lane's features (f = lane + 64 i), under
// the coalition whose presence test is `present(p)`.
template <class Present>
__device__ __forceinline__ void layer1(const GatDev& g, int64_t x, Present present, float (&out)[kGatSlots]) {
  const int lane = threadIdx.x & 63;
  float num[kGatSlots], den[kGatSlots];
#pragma unroll
  for (int i = 0; i < kGatSlots; ++i) {
    const int f = lane + 64 * i;
    if (f < g.nf) {
      const float ws = g.wself[x * g.H + f / g.F];
      num[i] = ws * g.z1[x * g.nf + f];
      den[i] = ws;
    } else {
      num[i] = 0.f;
      den[i] = 1.f;
    }
  }
  const int32_t p0 = g.dst_ptr[x], p1 = g.dst_ptr[x + 1];
  for (int32_t p = p0; p < p1; ++p) {
    if (!present(p)) continue;
    const int64_t u = g.esrc[p];
#pragma unroll
    for (int i = 0; i < kGatSlots; ++i) {
      const int f = lane + 64 * i;
      if (f < g.nf) {
        const float wp = g.w[static_cast<int64_t>(p) * g.H + f / g.F];
        num[i] += wp * g.z1[u * g.nf + f];
        den[i] += wp;
      }
    }
  }
#pragma unroll
  for (int i = 0; i < kGatSlots; ++i) {
    const int f = lane + 64 * i;
    out[i] = f < g.nf ? elu(num[i] / den[i] + g.b1[f]) : 0.f;
  }
}

// Dot product of a lane-distributed layer-1 output with a vector of nf (sum over the wave).
__device__ __forceinline__ float dot_nf(const GatDev& g, const float (&o)[kGatSlots], const float* v, int64_t stride) {
  const int lane = threadIdx.x & 63;
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < kGatSlots; ++i) {
    const int f = lane + 64 * i;
    if (f < g.nf) s += o[i] * v[f * stride];
  }
  return wave_sum_f(s);
}

// Layer-2 output at v for class c under a coalition (one wave): online
// softmax over the self loop and the present in-edges of v.
template <class Present>
__device__ float value_at_v(const GatDev& g, int32_t c, Present present) {
  float o[kGatSlots];
  layer1(g, 0, present, o);
  const float sdv = dot_nf(g, o, g.u2d, 1);
  float mx = leaky(dot_nf(g, o, g.u2s, 1) + sdv, g.slope);
  float sum = 1.f;
  float acc = dot_nf(g, o, g.W2 + c, g.C);
  for (int64_t e = 0; e < g.indeg_v; ++e) {
    if (!present(static_cast<int32_t>(e))) continue;
    const int64_t x = g.esrc[e];
    layer1(g, x, present, o);
    const float lx = leaky(dot_nf(g, o, g.u2s, 1) + sdv, g.slope);
    const float yx = dot_nf(g, o, g.W2 + c, g.C);
    if (lx > mx) {
      const float r = expf(mx - lx);
      sum = sum * r + 1.f;
      acc = acc * r + yx;
      mx = lx;
    } else {
      const float wx = expf(lx - mx);
      sum += wx;
      acc += wx * yx;
    }
  }
  return acc / sum + g.b2[c];
}

// f(empty) and f(E_c) for every class (one wave per class and end
// coalition), then the explained class and f_empty_full.  One workgroup.
__global__ void __launch_bounds__(1024) k_gat_ends(GatDev g, int32_t target_class, float* fef, int32_t* class_out,
                                                  float* scratch) {
  const int wv = threadIdx.x >> 6, nw = blockDim.x >> 6;
  for (int64_t t = wv; t < 2 * g.C; t += nw) {
    const int32_t c = static_cast<int32_t>(t % g.C);
    const bool full = t >= g.C;
    const float v = full ? value_at_v(g, c, [](int32_t) { return true; })
                         : value_at_v(g, c, [](int32_t) { return false; });
    if ((threadIdx.x & 63) == 0) scratch[t] = v;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int32_t c = target_class;
    if (c < 0) {
      c = 0;
      for (int32_t i = 1; i < g.C; ++i)
        if (scratch[g.C + i] > scratch[g.C + c]) c = i;
    }
    *g.cls = c;
    fef[0] = scratch[c];
    fef[1] = scratch[g.C + c];
    if (class_out) *class_out = c;
  }
}

// y[b] for coalition b: one wave per coalition.
__global__ void __launch_bounds__(kRowsWaves * 64) k_gat_rows(GatDev g, const uint64_t* __restrict__ masks,
                                                              int64_t k, int64_t wpr, const float* __restrict__ fef,
                                                              float* __restrict__ y) {
  const int64_t b = static_cast<int64_t>(blockIdx.x) * kRowsWaves + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (b >= k) return;
  const uint64_t* row = masks + b * wpr;
  auto present = [row](int32_t p) { return ((row[p >> 6] >> (p & 63)) & 1ull) != 0; };
  bool live = false;
  for (int64_t w = 0; w * 64 < g.indeg_v; ++w) {
    const int64_t n = g.indeg_v - w * 64;
    const uint64_t m = n >= 64 ? ~0ull : ((1ull << n) - 1ull);
    live |= (row[w] & m) != 0;
  }
  float v;
  if (!live) v = fef[0];   // no in-edge of v: the target alone (Sec. 3.4.1)
  else v = value_at_v(g, *g.cls, present);
  if ((threadIdx.x & 63) == 0) y[b] = v;
}

struct GatWs {
  float *z1, *ss1, *sd1, *w, *wself, *u2s, *u2d, *scratch;
  int32_t* cls;
};

GatWs gat_carve(gnnshap::Carver& c, const gnnshap_subgraph* sg, const gnnshap_gat* m) {
  const int64_t nf = static_cast<int64_t>(m->heads) * m->head_dim;
  GatWs w;
  w.z1 = c.take<float>(sg->num_nodes * nf);
  w.ss1 = c.take<float>(sg->num_nodes * m->heads);
  w.sd1 = c.take<float>(sg->num_dst * m->heads);
  w.w = c.take<float>(sg->num_edges * m->heads);
  w.wself = c.take<float>(sg->num_dst * m->heads);
  w.u2s = c.take<float>(nf);
  w.u2d = c.take<float>(nf);
  w.scratch = c.take<float>(2 * static_cast<int64_t>(m->num_classes));
  w.cls = c.take<int32_t>(1);
  return w;
}

int gat_check(const gnnshap_subgraph* sg, const gnnshap_gat* m) {
  if (!sg || !m) return gnnshap::fail(GNNSHAP_EINVAL, "null subgraph or model");
  if (sg->num_hops != 2) return gnnshap::fail(GNNSHAP_EINVAL, "the two-layer GAT needs a 2-hop subgraph");
  if (sg->num_edges < 1 || sg->num_dst < 1 || sg->num_nodes < sg->num_dst)
    return gnnshap::fail(GNNSHAP_EINVAL, "subgraph sizes are inconsistent");
  if (m->heads < 1 || m->head_dim < 1 || static_cast<int64_t>(m->heads) * m->head_dim > kGatMaxFeat)
    return gnnshap::fail(GNNSHAP_EINVAL, "heads * head_dim must be in [1, %d]", kGatMaxFeat);
  if (m->num_classes < 1 || m->num_classes > GNNSHAP_MAX_CLASSES)
    return gnnshap::fail(GNNSHAP_EINVAL, "num_classes out of range");
  if (!(m->negative_slope >= 0.0 && m->negative_slope < 1.0))
    return gnnshap::fail(GNNSHAP_EINVAL, "negative_slope must be in [0, 1)");
  if (!m->XW1 || !m->att_src1 || !m->att_dst1 || !m->W2 || !m->att_src2 || !m->att_dst2)
    return gnnshap::fail(GNNSHAP_EINVAL, "null model array");
  return GNNSHAP_OK;
}

}  // namespace

extern "C" int gnnshap_gat_eval_workspace(const gnnshap_subgraph* sg, const gnnshap_gat* m, int64_t k,
                                          size_t* bytes) {
  gnnshap::clear_error();
  if (!bytes || k < 1) return gnnshap::fail(GNNSHAP_EINVAL, "bad arguments");
  if (int st = gat_check(sg, m)) return st;
  gnnshap::Carver c(nullptr);
  gat_carve(c, sg, m);
  *bytes = c.bytes();
  return GNNSHAP_OK;
}

extern "C" int gnnshap_gat_eval_coalitions(const gnnshap_subgraph* sg, const gnnshap_gat* m, int32_t target_class,
                                           const uint64_t* masks, int64_t k, int64_t words_per_row, float* y,
                                           float* f_empty_full, int32_t* class_out, void* ws, size_t ws_bytes,
                                           void* stream) {
  GS_TRY_BEGIN
  gnnshap::clear_error();
  if (int st = gat_check(sg, m)) return st;
  if (!masks || !y || !f_empty_full || !ws || k < 1) return gnnshap::fail(GNNSHAP_EINVAL, "null argument or k < 1");
  if (!sg->node_gid || !sg->dst_ptr || !sg->edge_src) return gnnshap::fail(GNNSHAP_EINVAL, "null subgraph arrays");
  if (words_per_row != gnnshap::ceil_div(sg->num_edges, 64))
    return gnnshap::fail(GNNSHAP_EINVAL, "words_per_row != ceil(M/64)");
  if (target_class < -1 || target_class >= m->num_classes)
    return gnnshap::fail(GNNSHAP_EINVAL, "target_class out of range");
  gnnshap::Carver need(nullptr);
  gat_carve(need, sg, m);
  if (ws_bytes < need.bytes()) return gnnshap::fail(GNNSHAP_ECAPACITY, "GAT workspace needs %zu bytes", need.bytes());
  gnnshap::Carver cv(ws);
  const GatWs w = gat_carve(cv, sg, m);
  hipStream_t s = static_cast<hipStream_t>(stream);
  GatDev g{};
  g.gid = sg->node_gid;
  g.dst_ptr = sg->dst_ptr;
  g.esrc = sg->edge_src;
  g.n_nodes = sg->num_nodes;
  g.n1 = sg->num_dst;
  g.M = sg->num_edges;
  // hop-1 nodes are exactly v's in-neighbours, so v has hop_ptr[2] - 1 players
  g.indeg_v = sg->hop_ptr[2] - sg->hop_ptr[1];
  g.H = m->heads;
  g.F = m->head_dim;
  g.nf = m->heads * m->head_dim;
  g.C = m->num_classes;
  g.XW1 = m->XW1;
  g.att_src1 = m->att_src1;
  g.att_dst1 = m->att_dst1;
  g.b1 = m->b1;
  g.W2 = m->W2;
  g.att_src2 = m->att_src2;
  g.att_dst2 = m->att_dst2;
  g.b2 = m->b2;
  g.slope = static_cast<float>(m->negative_slope);
  g.z1 = w.z1;
  g.ss1 = w.ss1;
  g.sd1 = w.sd1;
  g.w = w.w;
  g.wself = w.wself;
  g.u2s = w.u2s;
  g.u2d = w.u2d;
  g.cls = w.cls;
  if (!g.b1 || !g.b2) return gnnshap::fail(GNNSHAP_EINVAL, "the GAT needs both biases (zero arrays for none)");
  k_gat_gather<<<gnnshap::grid_for(sg->num_nodes * g.nf, 256, 1024), 256, 0, s>>>(g);
  GS_LAUNCHED();
  k_gat_weights<<<gnnshap::grid_for(std::max<int64_t>(sg->num_dst * g.H, g.nf), 256, 256), 256, 0, s>>>(g);
  GS_LAUNCHED();
  {
    GS_TIMED("k_gat_ends", s);
    k_gat_ends<<<1, 1024, 0, s>>>(g, target_class, f_empty_full, class_out, w.scratch);
  }
  GS_LAUNCHED();
  {
    GS_TIMED("k_gat_rows", s);
    k_gat_rows<<<static_cast<unsigned>(gnnshap::ceil_div(k, kRowsWaves)), kRowsWaves * 64, 0, s>>>(
        g, masks, k, words_per_row, f_empty_full, y);
  }
  GS_LAUNCHED();
  return GNNSHAP_OK;
  GS_TRY_END
}
