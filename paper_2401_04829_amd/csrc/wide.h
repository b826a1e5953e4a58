// Internal interface of the coalition evaluation for GCNs with wide hidden
// layers on two hops (Sec. 3.4, GCN of Sec. 4.2): the masked aggregation of
// each layer at the nodes of H_1 as a contraction on bf16 MFMA over an exact
// split of the fp32 operand.  Two-layer models run it once (layer 1, then
// the explained class's column of W_2); three-layer models run it for layer
// 1 (full rows), a dense transform by W_2, then for layer 2 (with the
// coalitions' own rows for sources in H_1), in passes over the rows.
#pragma once

#include "common.h"

namespace gnnshap {

struct WideShape {
  int64_t M = 0, n_nodes = 0, n1 = 0, k = 0;
  int64_t n2 = 0;          // the target and its in-neighbours (nodes 0 .. n2 - 1; n2 = n1 with two hops)
  int64_t units_cap = 0;   // operand units (32 players each) of the contraction, upper bound
  int h = 0, C = 0;        // layer-1 width; classes
  int ntot = 0;            // 16-feature tiles of layer 1
  int nfb = 0;             // feature blocks (of at most four tiles) of layer 1
  int h2 = 0;              // three-layer models: layer-2 width (0: two layers)
  int ntot2 = 0, nfb2 = 0;
  int64_t pass = 0;        // three-layer models: contracted rows per pass
  bool agg3 = false;       // three hops (n2 < n1): layer 2 from A W_2 (launch_wide3_agg, launch_wide3_t)
};

// Whether the wide path evaluates a model: two or three layers over two
// hops, or three layers over three hops, hidden widths multiples of 16
// above 32.  H_1 (n1 nodes) is the set of nodes that players enter: the
// target and the first hop with two hops, and also the second hop with
// three; n2 counts the target and its in-neighbours.
bool wide_applies(int num_layers, int num_hops, const int32_t* dims);
WideShape wide_shape(int64_t M, int64_t n_nodes, int64_t n1, int64_t n2, int64_t k, const int32_t* dims,
                     int num_layers);

struct WideWs {
  int32_t* seg;       // n1 + 1: first operand unit of each node of H_1
  int32_t* spec_ptr;  // n1 + 1: players of each node whose source is in H_1
  int32_t* spec_e;    // M
  uint4* Zop;         // units_cap x ntot x 3 x 64: layer-1 A operands in bf16 parts (see the kernels)
  float* S;           // n1 x h: sum of the layer-1 operand rows of each node
  int32_t* deg;       // k x n1: in-degree of each node of H_1 under each evaluated row
  float* t;           // (nfb or nfb2) x k x n1: each node's last hidden output times the explained class's column
  float* hf;          // (n1 + 1) x h: layer 1 under the end coalitions (E_c at H_1, then empty at the target)
  float* hp;          // 4 x n1 x max(h, h2): partial sums of the players entering each node under E_c
  float* z2e;         // three layers: (n1 + 1) x h2: hf W_2
  float* hf2;         // three layers: (n1 + 1) x h2: layer 2 under the end coalitions
  uint4* Zop2;        // three layers: units_cap x ntot2 x 3 x 64: layer-2 A operands
  float* S2;          // three layers: n1 x h2
  float* H1;          // three layers: 2 pass x n1 x h: layer 1 of the pass's rows (complements after them)
  float* Z2;          // three layers: 2 pass x n1 x h2: H1 W_2 (agg3: 2 pass x n2 x h2, A3 W_2)
  float* A3;          // agg3: 2 pass x n2 x h: layer 2's sums at nodes 0 .. n2 - 1 before W_2
};
WideWs wide_carve(Carver& c, const WideShape& s);

// The end coalitions of a two-layer model: sp_y[c] = f_c(empty), sp_y[C +
// c] = f_c(E_c) for every class, then the explained class (target_class, or
// argmax f(E_c)) into ctl[0], class_out (may be null) and f_empty_full.
int launch_wide_ends(const WideShape& s, const WideWs& w, const gnnshap_subgraph* sg, const float* Zc, const float* b1,
                     const float* W2, const float* b2, int32_t target_class, float* sp_y, int32_t* ctl,
                     int32_t* class_out, float* f_empty_full, hipStream_t st);

// y[b] for rows b < k of `masks` (f(empty) for rows without an in-edge of
// the target), two-layer model.  Zc: n_nodes x h rows of X W_1 for the
// subgraph's nodes; ctl[0]: the explained class; fef[0]: f(empty).  pairs:
// rows b and b + k/2 are complements (the sampler's layout), so only the
// first half is contracted and the second half follows from it.
int launch_wide(const WideShape& s, const WideWs& w, const gnnshap_subgraph* sg, const uint64_t* masks, int64_t wpr,
                const float* Zc, const float* b1, const float* W2, const float* b2, const int32_t* ctl,
                const float* fef, bool pairs, float* y, hipStream_t st);

// The end coalitions of a three-layer model: launch_wide3_ends_l1 (layer 1
// into hf), then the caller's z2e = hf W_2, then launch_wide3_ends_l2 (layer
// 2, the output layer for every class and the explained class, as
// launch_wide_ends).
int launch_wide3_ends_l1(const WideShape& s, const WideWs& w, const gnnshap_subgraph* sg, const float* Zc1,
                         const float* b1, hipStream_t st);
int launch_wide3_ends_l2(const WideShape& s, const WideWs& w, const gnnshap_subgraph* sg, const float* Zc2,
                         const float* b2, const float* W3, const float* b3, int32_t target_class, float* sp_y,
                         int32_t* ctl, int32_t* class_out, float* f_empty_full, hipStream_t st);

// Three-layer model, in the order the caller queues them:
//   launch_wide3_prep    operand units, player lists, both layers' A
//                        operands (Zc1: X W_1 rows; Zc2: layer-2 input rows
//                        of the nodes outside H_1, constant) and sums, degrees
//   for each pass (rows r0 .. r0 + nloc - 1 of the contracted ones):
//     launch_wide3_l1    H1 of the pass's rows (and complements)
//     (the caller)       Z2 = H1 W_2
//     launch_wide3_l2    t from layer 2 with Z2 for the sources in H_1
//   launch_wide3_out     y from t (as the two-layer path's last step)
int launch_wide3_prep(const WideShape& s, const WideWs& w, const gnnshap_subgraph* sg, const uint64_t* masks,
                      int64_t wpr, const float* Zc1, const float* Zc2, bool pairs, hipStream_t st);
int launch_wide3_l1(const WideShape& s, const WideWs& w, const gnnshap_subgraph* sg, const uint64_t* masks,
                    int64_t wpr, int64_t r0, int64_t nloc, const float* Zc1, const float* b1, bool pairs,
                    hipStream_t st);
int launch_wide3_l2(const WideShape& s, const WideWs& w, const gnnshap_subgraph* sg, const uint64_t* masks,
                    int64_t wpr, int64_t r0, int64_t nloc, const float* b2, const float* W3, const int32_t* ctl,
                    bool pairs, hipStream_t st);
// Three hops (s.agg3), in place of the caller's Z2 = H1 W_2 and
// launch_wide3_l2: launch_wide3_agg (A3), the caller's Z2 = A3 W_2 (2 nloc
// n2 rows with pairs), launch_wide3_t (t at nodes 0 .. n2 - 1).
int launch_wide3_agg(const WideShape& s, const WideWs& w, const gnnshap_subgraph* sg, const uint64_t* masks,
                     int64_t wpr, int64_t r0, int64_t nloc, bool pairs, hipStream_t st);
int launch_wide3_t(const WideShape& s, const WideWs& w, const gnnshap_subgraph* sg, const uint64_t* masks,
                   int64_t wpr, int64_t r0, int64_t nloc, const float* b2, const float* W3, const int32_t* ctl,
                   bool pairs, hipStream_t st);
int launch_wide3_out(const WideShape& s, const WideWs& w, const gnnshap_subgraph* sg, const uint64_t* masks,
                     int64_t wpr, const float* b3, const int32_t* ctl, const float* fef, bool pairs, float* y,
                     hipStream_t st);

}  // namespace gnnshap
