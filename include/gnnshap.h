/*
 * gnnshap.h - C ABI of the GNNShap coalition-evaluation path for one AMD
 * Instinct MI355X (gfx950).
 *
 * GNNShap (Akkas & Azad, arXiv 2401.04829) explains the prediction of a GNN
 * for one target node v by a Shapley value for every directed edge of v's
 * pruned computational graph.  Alg. 1 of the paper has four steps; each has
 * an entry point here:
 *
 *   1. gnnshap_extract_subgraph   prune the l-hop computational graph (Sec. 3.2)
 *   2. gnnshap_plan_samples       size classes and weights (eq. 4-6, Alg. 2)
 *      gnnshap_sample_coalitions  coalition masks and weights (Alg. 3, App. C.1)
 *   3. gnnshap_eval_coalitions    masked GCN predictions (Sec. 3.4)
 *   4. gnnshap_solve_wls          constrained weighted least squares (eq. 2-3, Sec. 3.5)
 *
 * Conventions shared by every call:
 *   - "[dev]" pointers are device memory of the current HIP device, "[host]"
 *     pointers host memory.  Every buffer a call reads or writes is owned by
 *     the caller, and device scratch space comes from the *_workspace queries
 *     (the byte size of a caller-owned device buffer).  The library allocates
 *     no device memory of its own, but it keeps these resources from their
 *     first use until the process ends (never freed by a call):
 *       . page-locked host staging buffers, per calling host thread
 *         (hipHostMalloc), through which the batched calls' job tables reach
 *         the device and the batched extraction's sizes come back;
 *       . two side streams with their events per device and calling host
 *         thread, events marking each evaluated target, and one worker host
 *         thread per calling thread (gnnshap_explain_batch);
 *       . mapped page-locked stop flags, one per iterative solve in flight
 *         (at most 16 per calling thread), and two events per group of
 *         iterative solves in flight (at most 8 groups per calling thread);
 *       . a fixed 512 KiB device array per GPU, in the library's code
 *         object (gnnshap_sample_coalitions_noalloc);
 *       . a host cache of recent (M, p) sample plans.
 *   - `stream` is a hipStream_t (NULL = the default stream).  All device work
 *     is enqueued on it and is asynchronous, except where a call says it
 *     blocks: the extraction calls (they return sizes), and
 *     gnnshap_solve_wls and gnnshap_explain_batch when a system is solved
 *     iteratively (the host waits on the stream for each chunk's stopping
 *     test, so the call returns once the iteration has stopped).
 *   - Return value: a gnnshap_status.  No C++ exception crosses the ABI.  On
 *     GNNSHAP_EINVAL or GNNSHAP_ECAPACITY nothing is written except the sizes
 *     a call reports.  gnnshap_last_error() gives a thread-local message about
 *     the last failure.
 *   - All floating-point device data is fp32, row-major.
 */
#ifndef GNNSHAP_H
#define GNNSHAP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum gnnshap_status {
  GNNSHAP_OK = 0,
  GNNSHAP_EINVAL = 1,       /* invalid argument */
  GNNSHAP_ECAPACITY = 2,    /* a caller buffer or workspace is too small; sizes reported */
  GNNSHAP_EHIP = 3,         /* a HIP runtime call failed */
  GNNSHAP_ESINGULAR = 4,    /* reserved: the solver reports pivots through `info` */
  GNNSHAP_EUNSUPPORTED = 5  /* valid but outside what the library implements */
};

#define GNNSHAP_MAX_HOPS 8
#define GNNSHAP_MAX_LAYERS 8
#define GNNSHAP_MAX_CLASSES 1024

const char* gnnshap_status_str(int status);
const char* gnnshap_last_error(void);
int gnnshap_version(void); /* major*10000 + minor*100 + patch */

/* ------------------------------------------------------------------------ */
/* Graph: in-CSR of a simple directed graph (row = destination).            */
/* The sources of the edges u -> w are indices[indptr[w] .. indptr[w+1]),   */
/* ascending, without duplicates or self loops.                             */
/* ------------------------------------------------------------------------ */
typedef struct {
  int64_t num_nodes;
  int64_t num_edges;
  const int64_t* indptr;   /* [dev] num_nodes + 1 */
  const int32_t* indices;  /* [dev] num_edges */
} gnnshap_graph;

/* ------------------------------------------------------------------------ */
/* 1. Pruned computational graph (Sec. 3.2 and App. A; Fig. 2).             */
/*                                                                          */
/* dist(u) = length of the shortest directed path u -> ... -> v.  With l =  */
/* num_hops, the players are the edges whose message reaches v within l     */
/* layers: E_c = {(u -> w) : dist(w) <= l-1}; the nodes are V_c = {u :      */
/* dist(u) <= l}.  Local node ids sort V_c by (dist, global id): v is local */
/* node 0 and the nodes within j hops are the prefix [0, hop_ptr[j+1]).     */
/* Players are ordered by (local destination, source global id); the        */
/* players entering local node x are [dst_ptr[x], dst_ptr[x+1]) for         */
/* x < num_dst = hop_ptr[l] (the nodes within l-1 hops).  Players           */
/* 0 .. indeg(v)-1 are the in-edges of v.                                   */
/* ------------------------------------------------------------------------ */
typedef struct {
  int32_t num_hops;        /* in: l, 1 .. GNNSHAP_MAX_HOPS */
  int32_t reserved;
  int64_t cap_nodes;       /* in: capacity of node_gid (and of dst_ptr minus one) */
  int64_t cap_edges;       /* in: capacity of edge_src, edge_dst, edge_gid */
  int32_t* node_gid;       /* [dev] out: global id of local node i, i < num_nodes */
  int32_t* dst_ptr;        /* [dev] out: num_dst + 1 player offsets */
  int32_t* edge_src;       /* [dev] out: local source of player p */
  int32_t* edge_dst;       /* [dev] out: local destination of player p */
  int64_t* edge_gid;       /* [dev] out: position of player p in indices[] */
  int64_t num_nodes;       /* out: |V_c| */
  int64_t num_edges;       /* out: M = |E_c| (number of players) */
  int64_t num_dst;         /* out: |H_{l-1}| */
  int64_t hop_ptr[GNNSHAP_MAX_HOPS + 2]; /* out: hop_ptr[0..l+1] */
} gnnshap_subgraph;

/* Bytes of device workspace for graphs of `num_nodes` nodes. */
int gnnshap_extract_workspace(int64_t num_nodes, size_t* bytes);

/* Extracts the computational graph of `target`.  `ws` must be zero-filled
 * before its first use; every call that returns (with any status) leaves it
 * zero-filled again, so it can be reused across calls without clearing.
 * BLOCKS the host: the sizes (num_nodes, num_edges, ...) are returned in *sg
 * after a synchronisation of `stream`.  If cap_nodes or cap_edges is too
 * small, returns GNNSHAP_ECAPACITY with the required sizes in *sg and writes
 * no output array.  EINVAL: null pointers, target out of range, bad hops. */
int gnnshap_extract_subgraph(const gnnshap_graph* g, int64_t target,
                             gnnshap_subgraph* sg, void* ws, size_t ws_bytes,
                             void* stream);

/* ------------------------------------------------------------------------ */
/* 2. Coalition sampling (Sec. 3.3, eq. 4-6, Alg. 2-3, App. C.1).           */
/*                                                                          */
/* Size class c (1 <= c <= M/2) holds the coalitions of size c and, through */
/* complements, of size M-c; omega_c = kappa_c (M-1)/(c(M-c)) with kappa_c  */
/* = 2, or 1 for the middle class c = M/2 of even M (eq. 4).  Classes are   */
/* enumerated in ascending c while their eq. 5 share of the pairs left is   */
/* at least their number of coalitions (Sec. 3.3.1 surplus redistribution); */
/* the remaining pairs are spread over the other classes in proportion to   */
/* omega (eq. 5), largest remainder, ties to the smaller c.  Enumerated     */
/* rows carry the Kernel-SHAP weight (eq. 3) divided by sum(rho); all random */
/* rows carry one common weight (Alg. 2).  Rows [0, k/2) are                */
/* representatives: enumerated classes first (lexicographic rank order),    */
/* then random classes (Floyd's algorithm on Philox4x32-10 draws: draw s of */
/* row i uses counter (s/4, i, stream_lo, stream_hi), key (seed_lo,         */
/* seed_hi), word s%4, mapped to [0, j] as (u*(j+1))>>32).  Row i + k/2 is   */
/* the complement of row i.                                                 */
/*                                                                          */
/* Mask layout: row b is words_per_row = ceil(M/64) uint64 words; player j  */
/* is bit j%64 of word b*words_per_row + j/64; padding bits are zero.       */
/* ------------------------------------------------------------------------ */
typedef struct {
  int32_t size;            /* coalition size c of the representative rows */
  int32_t full;            /* 1 = enumerated in rank order, 0 = random */
  int64_t row_begin;       /* first representative row of the class */
  int64_t row_count;       /* number of representative rows */
  double weight;           /* weight of each row of the class and of its complement */
} gnnshap_class;

typedef struct {
  int64_t num_players;     /* in: M >= 2 */
  int64_t num_samples;     /* in: p >= 2, even (the budget) */
  uint64_t seed;           /* in: Philox key */
  uint64_t stream_id;      /* in: Philox stream (e.g. the target's global id) */
  int64_t num_rows;        /* out: k <= p rows actually produced (even) */
  int64_t words_per_row;   /* out: ceil(M/64) */
  int64_t num_classes;     /* out: number of gnnshap_class records */
  int64_t random_begin;    /* out: first random representative row */
  double full_fraction;    /* out: total weight of the enumerated rows */
  double random_weight;    /* out: weight of every random row (0 if none) */
  int64_t iterative_threshold; /* in: systems of more players than this are solved
                                  iteratively by gnnshap_solve_wls (Sec. 3.5); 0 or
                                  negative = 5000, the paper's switch.  Kept by
                                  gnnshap_plan_samples; gnnshap_plan_batch sets 0. */
} gnnshap_sample_plan;

/* Host-only, pure, thread-safe (plans of recent (M, p) pairs are kept and
 * reused).  Fills *plan's outputs and classes[0 .. num_classes); the inputs
 * (num_players, num_samples, seed, stream_id, iterative_threshold) are kept.
 * If `classes` is NULL or cap_classes < num_classes, returns
 * GNNSHAP_ECAPACITY with the outputs of *plan filled.  EINVAL: M < 2, odd
 * or non-positive p, or more than 2^31 rows. */
int gnnshap_plan_samples(gnnshap_sample_plan* plan, gnnshap_class* classes,
                         int64_t cap_classes);

/* Bytes of device workspace for gnnshap_sample_coalitions. */
int gnnshap_sample_workspace(const gnnshap_sample_plan* plan, size_t* bytes);

/* Writes masks[num_rows * words_per_row] and weights[num_rows] (fp32, the
 * rounding of the fp64 class weight).  `classes` is the host table filled
 * by gnnshap_plan_samples; it is copied to `ws` on `stream` and must stay
 * unchanged until that copy has run.  EUNSUPPORTED: M too large for the
 * on-chip row buffer (M > 131072). */
int gnnshap_sample_coalitions(const gnnshap_sample_plan* plan,
                              const gnnshap_class* classes,
                              uint64_t* masks, float* weights,
                              void* ws, size_t ws_bytes, void* stream);

/* gnnshap_sample_coalitions without a workspace, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation).  The class table is copied on
 * `stream` into a fixed array of the library (512 KiB, 16384 records, one
 * per GPU, held until the process ends) instead of the caller's workspace;
 * the call allocates nothing.  Every call on a GPU shares that GPU's array:
 * calls that overlap on one GPU (different streams or host threads) race and
 * must be ordered by the caller.  Same outputs, bit for bit, and errors as
 * gnnshap_sample_coalitions; ECAPACITY if the plan has more than 16384 class
 * records (a plan has at most M/2; 30,000 players and 100,000 samples give
 * about 13,200); EHIP if the array's device address cannot be obtained. */
int gnnshap_sample_coalitions_noalloc(const gnnshap_sample_plan* plan,
                                      const gnnshap_class* classes,
                                      uint64_t* masks, float* weights,
                                      void* stream);

/* ------------------------------------------------------------------------ */
/* 3. Masked GCN predictions (Sec. 3.4, GCN of Sec. 4.2).                   */
/*                                                                          */
/* For coalition S: A_S[w,u] = 1 iff (u -> w) in S; deg_S(x) = 1 + in-degree */
/* of x under S; Ahat_S = D^-1/2 (A_S + I) D^-1/2; H^0 = X[V_c];            */
/* H^l = Ahat_S H^(l-1) W_l + b_l with ReLU after every layer but the last; */
/* y = H^L[v, target_class].  Coalitions without an in-edge of v are not    */
/* evaluated: their value is f(empty) (Sec. 3.4.1, exact).                  */
/* ------------------------------------------------------------------------ */
typedef struct {
  int32_t num_layers;            /* L, 1 .. GNNSHAP_MAX_LAYERS */
  int32_t reserved;
  const int32_t* dims;           /* [host] L + 1 widths: dims[0] = feature width d,
                                    dims[L] = number of classes C */
  const float* const* W;         /* [host] L [dev] pointers; W_l is dims[l] x dims[l+1] */
  const float* const* b;         /* [host] L [dev] pointers, or NULL entries / NULL = zero bias */
  const float* XW1;              /* [dev] optional num_nodes x dims[1]: X W_1 for every node of the
                                    graph (gnnshap_transform_features); NULL = computed from X */
} gnnshap_gcn;

/* Z = X W for every node (fp32; X [dev] n x d, W [dev] d x h, Z [dev] n x h, row-major).
 * The first GCN layer transforms each node's features independently of the
 * coalition (Sec. 3.4.2: the coalitions of a batch share the node features),
 * so X W_1 is computed once per graph and model and passed as
 * gnnshap_gcn.XW1; each explanation then gathers the rows of its subgraph. */
int gnnshap_transform_features(const float* X, int64_t n, int32_t d, const float* W, int32_t h,
                               float* Z, void* stream);

/* Bytes of device workspace for evaluating k coalitions of subgraph sg. */
int gnnshap_eval_workspace(const gnnshap_subgraph* sg, const gnnshap_gcn* m,
                           int64_t k, size_t* bytes);

/* y[b] = f(S_b) for b < k.  sg is a subgraph as gnnshap_extract_subgraph
 * lays it out (its node and player order is relied on).  X is the [dev]
 * feature matrix of the whole graph (num_nodes x dims[0]).  target_class >= 0 selects the explained logit;
 * -1 selects argmax_c f(E_c)[c] (ties to the lowest c), computed on the
 * device and written to *class_out if class_out is not NULL ([dev] int32).
 * f_empty_full[0] = f(empty), f_empty_full[1] = f(E_c) ([dev] 2 floats). */
int gnnshap_eval_coalitions(const gnnshap_subgraph* sg, const gnnshap_gcn* m,
                            const float* X, int32_t target_class,
                            const uint64_t* masks, int64_t k,
                            int64_t words_per_row, float* y,
                            float* f_empty_full, int32_t* class_out,
                            void* ws, size_t ws_bytes, void* stream);

/* gnnshap_eval_coalitions for masks in the sampler's layout (Alg. 2 pairs
 * each sampled coalition with its complement, App. C.1): k is even and row
 * b + k/2 is the complement of row b within the M player bits for every
 * b < k/2, as gnnshap_sample_coalitions writes them (the call relies on it
 * and does not check it).  Same arguments, workspace and errors as
 * gnnshap_eval_coalitions (EINVAL also for odd k).  Two-layer models with a
 * wide hidden layer then contract only the first half of the rows: the
 * complement's masked sum is the sum over all players minus the row's. */
int gnnshap_eval_sampled_coalitions(const gnnshap_subgraph* sg, const gnnshap_gcn* m,
                                    const float* X, int32_t target_class,
                                    const uint64_t* masks, int64_t k,
                                    int64_t words_per_row, float* y,
                                    float* f_empty_full, int32_t* class_out,
                                    void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* 4. Constrained Kernel-SHAP least squares (eq. 2-3, Alg. 1, Sec. 3.5).    */
/*                                                                          */
/* phi = argmin sum_b w_b (y_b - f(empty) - m_b . phi)^2 subject to         */
/* sum(phi) = f(E_c) - f(empty) (efficiency; eq. 3's infinite weights at    */
/* the empty and full coalitions), over the rows of a plan.  Solved as the  */
/* projected system (P G P + gamma 11^T/M) psi = P(r - Delta/M G 1),        */
/* phi = Delta/M + psi, P = I - 11^T/M, with G = M^T W M built from exact   */
/* integer coalition counts and factored by Cholesky.                       */
/* ------------------------------------------------------------------------ */

/* Bytes of device workspace for a plan. */
int gnnshap_solve_workspace(const gnnshap_sample_plan* plan, size_t* bytes);

/* phi[M] from the plan's masks, the predictions y[k] and f_empty_full[2]
 * (all [dev]).  `classes` as for gnnshap_sample_coalitions.  *info ([dev]
 * int32) receives 0, or j > 0 if the j-th pivot (1-based) of the Cholesky
 * factorisation was not positive (phi is then not meaningful; this happens
 * when the sampled rows do not determine phi).
 * Systems of more than plan->iterative_threshold players (default 5000) are
 * not factored: conjugate gradients run on the projected normal
 * equations, applying the masks and their transpose straight from the bits
 * (Sec. 3.5 fits large systems iteratively), until the residual falls to
 * 1e-6 of its initial norm; *info is then 0, or M + 1 if that did not happen
 * within 4000 iterations, the iteration broke down, or the plan has no
 * enumerated class and fewer than M - 1 random rows (then the rows cannot
 * determine phi).  Other rank deficiencies are not detected on that path:
 * the residual can still fall and phi is then one of many minimisers.  That path waits on
 * `stream` for its stopping test (the call returns once the iteration has
 * stopped; the write of phi is still queued). */
int gnnshap_solve_wls(const gnnshap_sample_plan* plan,
                      const gnnshap_class* classes, const uint64_t* masks,
                      const float* y, const float* f_empty_full, float* phi,
                      int32_t* info, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* 5. Many targets per launch sequence (Alg. 1 for each of n targets).      */
/*                                                                          */
/* The explanations of different targets are independent (Alg. 1 runs per  */
/* target node); these calls run each step for a whole batch of targets in  */
/* one launch, so that targets with small computational graphs fill the     */
/* GPU together.  Every output equals, bit for bit, what the single-target  */
/* calls above give for the same arguments.                                 */
/* ------------------------------------------------------------------------ */

/* Bytes of device workspace for gnnshap_extract_batch on a graph of
 * num_nodes nodes and n targets. */
int gnnshap_extract_batch_workspace(int64_t num_nodes, int64_t n, size_t* bytes);

/* gnnshap_extract_subgraph for targets[0 .. n) ([host] int64) into sgs[0 .. n)
 * ([host] array; each entry has its own num_hops, capacities and [dev]
 * output arrays, as for the single call).  One workgroup per target, one
 * host synchronisation for the batch; `ws` zero-filled before first use,
 * after which every call leaves it ready for the next batch call (of any
 * n up to the size it was made for).  Sizes are filled in for every target; if any target
 * does not fit its capacities, returns GNNSHAP_ECAPACITY (the targets that
 * fit are complete).  EUNSUPPORTED: graphs of more than 2^18 nodes (use the
 * single-target call there).  EINVAL as for the single call. */
int gnnshap_extract_batch(const gnnshap_graph* g, const int64_t* targets, int64_t n,
                          gnnshap_subgraph* sgs, void* ws, size_t ws_bytes, void* stream);

/* gnnshap_extract_batch in two halves, so that a caller can queue the next
 * batch's extraction before the current batch's explanation and wait for
 * the sizes later.  _launch validates the arguments and queues the
 * extraction on `stream`, whose kernel writes the sizes straight into
 * page-locked host memory (same arguments and errors as gnnshap_extract_batch, except
 * that it never reports ECAPACITY for the subgraphs); _finish waits for
 * those sizes and fills them into sgs[0 .. n) (the same n and sgs array),
 * returning OK or ECAPACITY as gnnshap_extract_batch does.  The [dev]
 * outputs are complete when _finish returns.  Each host thread has at most
 * one launched extraction: _launch returns EINVAL while one is not
 * finished, _finish EINVAL when none is launched (or n differs).  `ws` and
 * the output arrays must not be touched between the two calls. */
int gnnshap_extract_batch_launch(const gnnshap_graph* g, const int64_t* targets, int64_t n,
                                 gnnshap_subgraph* sgs, void* ws, size_t ws_bytes, void* stream);
int gnnshap_extract_batch_finish(gnnshap_subgraph* sgs, int64_t n);

/* Host only: fills sgs[0 .. n) for outputs packed by target, as rows of
 * [dev] node_gid[n][cap_nodes], dst_ptr[n][cap_nodes + 1],
 * edge_src[n][cap_edges], edge_dst[n][cap_edges] (int32) and
 * edge_gid[n][cap_edges] (int64); every entry gets num_hops and the two
 * capacities, and zero sizes. */
int gnnshap_subgraph_batch_init(gnnshap_subgraph* sgs, int64_t n, int32_t num_hops, int64_t cap_nodes,
                                int64_t cap_edges, int32_t* node_gid, int32_t* dst_ptr, int32_t* edge_src,
                                int32_t* edge_dst, int64_t* edge_gid);

/* Host only, pure: gnnshap_plan_samples for each target of a batch.
 * plans[t] gets num_players = sgs[t].num_edges, num_samples, seed,
 * stream_id = stream_ids[t] ([host] int64, e.g. the target's global id)
 * and the outputs; the n class tables go to classes[] concatenated in
 * target order, *num_classes records in all.  totals ([host] int64[3], may
 * be NULL) receives the sizes of gnnshap_explain_batch's packed outputs:
 * sum_t k_t * words_per_row_t, sum_t k_t and sum_t M_t.  If `classes` is
 * NULL or cap_classes < *num_classes, returns GNNSHAP_ECAPACITY with plans,
 * *num_classes and totals filled.  EINVAL as for the single call, naming
 * the target. */
int gnnshap_plan_batch(const gnnshap_subgraph* sgs, const int64_t* stream_ids, int64_t n,
                       int64_t num_samples, uint64_t seed, gnnshap_sample_plan* plans,
                       gnnshap_class* classes, int64_t cap_classes, int64_t* num_classes,
                       int64_t* totals);

/* Bytes of device workspace for gnnshap_explain_batch. */
int gnnshap_explain_batch_workspace(const gnnshap_subgraph* sgs, const gnnshap_sample_plan* plans,
                                    int64_t n, const gnnshap_gcn* m, size_t* bytes);

/* Sampling, predictions and least squares of n targets.  sgs[t] ([host]) is
 * target t's extracted subgraph and plans[t] ([host]) its plan (from
 * gnnshap_plan_samples, num_players = sgs[t].num_edges); `classes` [host] is
 * the concatenation of the n class tables in target order (copied on
 * `stream`; keep it unchanged until then).  Outputs ([dev]) are packed in
 * target order:
 *   masks    rows of target t start at word sum_{s<t} k_s * words_per_row_s;
 *   weights, y   start at sum_{s<t} k_s;
 *   phi      starts at sum_{s<t} M_s;
 *   f_empty_full[2t .. 2t+1], class_out[t] (may be NULL), info[t].
 * X, target_class and the model as for gnnshap_eval_coalitions.  Two-layer
 * models with X W_1 given and one-workgroup systems run batched; other
 * targets go through the single-target kernels in the same sequence.
 * Systems factored by the multi-block Cholesky are set up one by one as
 * their coalition values are queued and factored and solved in runs of up
 * to 24 (one launch per step of the factorisation for the whole run).
 * Systems solved iteratively (more players than their plan's
 * iterative_threshold) run in two groups of up to three on the library's
 * side streams, each group advancing its systems together (one launch per
 * pass of the iteration for the whole group); a system joins a group once
 * its coalition values are computed.  The call returns once every
 * iteration has stopped (it polls the groups' events); the last writes of
 * phi and info are still queued, ordered before later work on `stream`.
 * EUNSUPPORTED: more than 65535 targets or M > 131072. */
int gnnshap_explain_batch(const gnnshap_subgraph* sgs, const gnnshap_sample_plan* plans,
                          const gnnshap_class* classes, int64_t n, const gnnshap_gcn* m,
                          const float* X, int32_t target_class, uint64_t* masks, float* weights,
                          float* y, float* f_empty_full, int32_t* class_out, float* phi,
                          int32_t* info, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* 6. Fidelity of an explanation (eq. 7-8, Sec. 4.3; protocol of Sec. 4.6). */
/*                                                                          */
/* Importance of a player is |phi| (Sec. 2.3), larger first, equal values   */
/* by lower player index.  G_S = all players but the floor(s M) least       */
/* important (sparsity s); G_{C\S} = all but the min(k, M) most important.  */
/* f is the explained output (the class logit, as for the coalitions).     */
/* ------------------------------------------------------------------------ */

/* The two coalitions: masks[0 .. wpr) = G_S, masks[wpr .. 2 wpr) = G_{C\S}
 * (wpr = ceil(M/64) words each, the mask layout of section 2) for phi [dev]
 * float[M]; masks [dev].  EINVAL: M < 1, sparsity outside [0, 1],
 * top_k < 0. */
int gnnshap_fidelity_masks(const float* phi, int64_t M, double sparsity, int64_t top_k, uint64_t* masks,
                           void* stream);

/* Bytes of device workspace for gnnshap_fidelity on subgraph sg. */
int gnnshap_fidelity_workspace(const gnnshap_subgraph* sg, const gnnshap_gcn* m, size_t* bytes);

/* One target's fidelity terms: out[0] = |f(G_C) - f(G_S)| (its term of
 * eq. 7), out[1] = |f(G_C) - f(G_{C\S})| (eq. 8), out[2] = f(G_C) ([dev]
 * 3 floats).  phi ([dev] float[M], M = sg->num_edges) are the explanation's
 * values; NaN values order unspecified.  G_S and G_{C\S} are written as two
 * coalitions and evaluated by gnnshap_eval_coalitions (target_class as
 * there: -1 = the predicted class on G_C).  EINVAL: sparsity outside
 * [0, 1], top_k < 0, a subgraph without players; ECAPACITY: workspace. */
int gnnshap_fidelity(const gnnshap_subgraph* sg, const gnnshap_gcn* m, const float* X, int32_t target_class,
                     const float* phi, double sparsity, int64_t top_k, float* out, void* ws, size_t ws_bytes,
                     void* stream);

/* eq. 7 and eq. 8 over n targets: avg[0] = mean of terms[t * stride],
 * avg[1] = mean of terms[t * stride + 1] (all [dev]; fp64 sums in a fixed
 * order).  EINVAL: n < 1 or stride < 2. */
int gnnshap_fidelity_average(const float* terms, int64_t n, int64_t stride, float* avg, void* stream);

/* ------------------------------------------------------------------------ */
/* 7. Coalition values of a two-layer GAT (App. E).                         */
/*                                                                          */
/* A coalition keeps its edges and every self loop.  Layer 1: `heads`       */
/* attention heads of width head_dim (Velickovic et al. 2018: z = X W_1,    */
/* e_h(u -> x) = LeakyReLU(a_src,h . z_h[u] + a_dst,h . z_h[x]), softmax    */
/* over the edges into x present in the coalition and the self loop,        */
/* out_h[x] = sum alpha z_h[u]), heads concatenated, plus b_1, then ELU.    */
/* Layer 2: one head of width num_classes on the layer-1 outputs, plus b_2. */
/* The softmax is renormalised under each coalition: only present edges     */
/* compete.  y = the layer-2 output at the target for the explained class.  */
/* The subgraph must have num_hops = 2 (players = edges into H_1).          */
/* ------------------------------------------------------------------------ */
typedef struct {
  int32_t heads;                 /* layer-1 heads, heads * head_dim <= 256 */
  int32_t head_dim;
  int32_t num_classes;           /* C, layer-2 width */
  int32_t reserved;
  const float* XW1;              /* [dev] num_nodes x heads*head_dim: X W_1 for every node
                                    (gnnshap_transform_features); required */
  const float* att_src1;         /* [dev] heads x head_dim */
  const float* att_dst1;         /* [dev] heads x head_dim */
  const float* b1;               /* [dev] heads*head_dim */
  const float* W2;               /* [dev] heads*head_dim x C */
  const float* att_src2;         /* [dev] C */
  const float* att_dst2;         /* [dev] C */
  const float* b2;               /* [dev] C */
  double negative_slope;         /* LeakyReLU slope of the attention logits, in [0, 1) (0.2) */
} gnnshap_gat;

/* Bytes of device workspace for evaluating k coalitions of sg with model m. */
int gnnshap_gat_eval_workspace(const gnnshap_subgraph* sg, const gnnshap_gat* m, int64_t k, size_t* bytes);

/* y[b] = f(S_b) for b < k under the GAT (outputs, classes and pruning as for
 * gnnshap_eval_coalitions: a coalition without an in-edge of the target has
 * the value f(empty)).  EINVAL: num_hops != 2, bad sizes or model arrays,
 * target_class out of range; ECAPACITY: workspace. */
int gnnshap_gat_eval_coalitions(const gnnshap_subgraph* sg, const gnnshap_gat* m, int32_t target_class,
                                const uint64_t* masks, int64_t k, int64_t words_per_row, float* y,
                                float* f_empty_full, int32_t* class_out, void* ws, size_t ws_bytes, void* stream);

/* Bytes of device workspace for gnnshap_gat_explain_batch. */
int gnnshap_gat_explain_batch_workspace(const gnnshap_subgraph* sgs, const gnnshap_sample_plan* plans, int64_t n,
                                        const gnnshap_gat* m, size_t* bytes);

/* gnnshap_explain_batch for the two-layer GAT (App. E): sampling, the
 * coalition values of gnnshap_gat_eval_coalitions for every target (one
 * launch sequence per target, in the batch's order) and the least squares,
 * with the same arguments, outputs, layout, streams and blocking as
 * gnnshap_explain_batch (m->XW1 replaces X).  Every output equals, bit for
 * bit, what the single-target calls give. */
int gnnshap_gat_explain_batch(const gnnshap_subgraph* sgs, const gnnshap_sample_plan* plans,
                              const gnnshap_class* classes, int64_t n, const gnnshap_gat* m, int32_t target_class,
                              uint64_t* masks, float* weights, float* y, float* f_empty_full, int32_t* class_out,
                              float* phi, int32_t* info, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Diagnostics: HIP-event timing of one kernel.                             */
/* ------------------------------------------------------------------------ */

/* Which solver the plan's system takes: *path = 1 if one workgroup factors
 * and solves it (M <= 192), 2 if it is factored panel by panel by small
 * workgroups (192 < M <= 448), 0 if it takes the multi-block Cholesky, 3 if
 * it is solved iteratively (M above plan->iterative_threshold; the
 * iterative path needs a different workspace, so the workspace query must
 * see the same threshold as the solve). */
int gnnshap_solve_info(const gnnshap_sample_plan* plan, int32_t* path);

/* Arms timing for the kernels whose name starts with `kernel_name` (e.g.
 * "k_solve_mid", "k_eval_l2"): every later launch of such a kernel, from
 * any entry point, is bracketed by two HIP events recorded on the launch's
 * own stream.  EINVAL if the name is empty or timing is already armed. */
int gnnshap_timing_begin(const char* kernel_name);

/* Disarms timing, waits for the recorded events and returns the summed
 * kernel time in milliseconds and the number of timed launches.  Timing
 * adds two event records per timed launch; not for concurrent use from
 * several host threads. */
int gnnshap_timing_end(double* total_ms, int64_t* launches);

/* The iterative solves (Sec. 3.5) run since the last gnnshap_timing_begin,
 * in the order they ran: records[6 i .. 6 i + 5] = players, mask words per
 * row, random representative rows, iterations (the iterations whose products
 * did work; up to seven more queued launches of each kernel find the solve
 * stopped and return at once), random rows kept as player lists (the first
 * ones, small coalitions), the players in those lists.  *count receives the
 * number of records; ECAPACITY if cap is smaller (cap counts records).
 * Diagnostics for measurements, like the timing calls. */
int gnnshap_timing_solves(int64_t* records, int64_t cap, int64_t* count);

#ifdef __cplusplus
}
#endif

#endif /* GNNSHAP_H */
