// Internal interface of the coalition evaluation for two-layer GCNs with a
// wide hidden layer (Sec. 3.4, GCN of Sec. 4.2): layer 1 at the nodes of H_1
// as a masked contraction on fp32 MFMA.
#pragma once

#include "common.h"

namespace gnnshap {

struct WideShape {
  int64_t M = 0, n_nodes = 0, n1 = 0, k = 0;
  int64_t units_cap = 0;   // operand units (16 players each) of the layer-1 contraction, upper bound
  int h = 0, C = 0;
  int ntot = 0;            // 16-feature tiles of the hidden layer
  int nfb = 0;             // feature blocks of at most eight tiles
};

// Whether the wide path evaluates a model: two layers, two hops (H_1 is then
// every node with players entering it), hidden width a multiple of 16 above 32.
bool wide_applies(int num_layers, int num_hops, int h);
WideShape wide_shape(int64_t M, int64_t n_nodes, int64_t n1, int64_t k, int h, int C);

struct WideWs {
  int32_t* seg;       // n1 + 1: first operand unit of each node of H_1
  int32_t* spec_ptr;  // n1 + 1: players of each node whose source is in H_1
  int32_t* spec_e;    // M
  uint4* Zop;         // units_cap x ntot x 3 x 64: A operands in bf16 parts (see the kernels)
  float* S;           // n1 x h: sum of the operand rows of each node
  int32_t* deg;       // k x n1: in-degree of each node of H_1 under each evaluated row
  float* t;           // nfb x k x n1: each node's layer-1 output times the explained class's W_2 column
  float* hf;          // (n1 + 1) x h: layer 1 under the end coalitions (E_c at H_1, then empty at the target)
  float* hp;          // 4 x n1 x h: partial sums of the players entering each node under E_c
};
WideWs wide_carve(Carver& c, const WideShape& s);

// The end coalitions: sp_y[c] = f_c(empty), sp_y[C + c] = f_c(E_c) for every
// class, then the explained class (target_class, or argmax f(E_c)) into
// ctl[0], class_out (may be null) and f_empty_full.
int launch_wide_ends(const WideShape& s, const WideWs& w, const gnnshap_subgraph* sg, const float* Zc, const float* b1,
                     const float* W2, const float* b2, int32_t target_class, float* sp_y, int32_t* ctl,
                     int32_t* class_out, float* f_empty_full, hipStream_t st);

// y[b] for rows b < k of `masks` (f(empty) for rows without an in-edge of
// the target).  Zc: n_nodes x h rows of X W_1 for the subgraph's nodes;
// ctl[0]: the explained class; fef[0]: f(empty).  pairs: rows b and b + k/2
// are complements (the sampler's layout), so only the first half is
// contracted and the second half follows from it.
int launch_wide(const WideShape& s, const WideWs& w, const gnnshap_subgraph* sg, const uint64_t* masks, int64_t wpr,
                const float* Zc, const float* b1, const float* W2, const float* b2, const int32_t* ctl,
                const float* fef, bool pairs, float* y, hipStream_t st);

}  // namespace gnnshap
