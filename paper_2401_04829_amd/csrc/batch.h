// Internal interface of the multi-target path: per-target job records that
// batched kernels read with blockIdx.y / blockIdx.z = target, and the
// launchers each stage exports to the batch driver.
#pragma once

#include "common.h"

namespace gnnshap {

// ---- sampling ---------------------------------------------------------------------------
struct SampleJob {
  const gnnshap_class* cls;  // device copy of the class table
  int64_t ncls, half, M, wpr;
  uint32_t seed_lo, seed_hi, st_lo, st_hi;
  uint64_t* masks;
  float* weights;
  int64_t blk0, rpb;         // first workgroup of the job in the launch, rows per workgroup
};
// Fills blk0 and rpb of jobs[0 .. n) (rows per workgroup inversely
// proportional to a row's cost, so that the workgroups of large and small
// targets take about as long) and returns the number of workgroups.
int64_t plan_sample_batch(SampleJob* jobs, int64_t n);
// Samples every job's rows: one workgroup per `rpb` rows of a job.
int launch_sample_batch(const SampleJob* jobs, int64_t n, int64_t blocks, int64_t max_wpr, hipStream_t s);

// ---- evaluation (two-layer GCN, one pass per target) -------------------------------------
struct EvalJob {
  const int32_t* node_gid;
  const int32_t* dst_ptr;
  const int32_t* edge_src;
  int64_t n_nodes, n_dst, n1, M, wpr, k;
  const uint64_t* masks;
  float* y;
  float* fef;
  int32_t* cls_out;
  // workspace
  int32_t* ctl;
  uint64_t* sp_masks;
  int32_t* sp_rows;
  float* sp_y;
  int32_t* live_rows;
  uint8_t* live_flag;
  float* Zc1;
  int32_t rows_ok;     // the main pass takes the one-thread-per-coalition kernel
};
struct EvalModel {
  const float* XW1;
  const float* b1;
  const float* W2;
  const float* b2;
  int h, C;
  int32_t target_class;
};
// gnnshap_eval_coalitions for masks in the sampler's layout (pairs = rows b
// and b + k/2 are complements; some paths then contract half of the rows).
int eval_coalitions_impl(const gnnshap_subgraph* sg, const gnnshap_gcn* m, const float* X, int32_t target_class,
                         const uint64_t* masks, int64_t k, int64_t words_per_row, float* y, float* f_empty_full,
                         int32_t* class_out, void* ws, size_t ws_bytes, void* stream, bool pairs);
// Whether one target can go through the batched evaluation, and the bytes of
// its workspace slice.
bool eval_batchable(const gnnshap_subgraph* sg, const gnnshap_gcn* m, int64_t k);
size_t eval_slice_bytes(const gnnshap_subgraph* sg, const gnnshap_gcn* m, int64_t k);
// Carves job.ctl .. job.Zc1 from a slice.
void eval_carve_slice(void* base, const gnnshap_subgraph* sg, const gnnshap_gcn* m, int64_t k, EvalJob* job);
// LDS of a target's one-thread-per-coalition main pass, 0 if it does not take it.
size_t eval_rows_lds(const gnnshap_subgraph* sg, const gnnshap_gcn* m);
int launch_eval_batch(const EvalJob* jobs, int64_t n, const EvalModel& md, int64_t max_nodes, int64_t max_ndst,
                      int64_t max_n1, int64_t max_wpr, int64_t max_k, int64_t rows_jobs, size_t rows_lds,
                      hipStream_t s);

// ---- least squares (one-workgroup systems) -----------------------------------------------
struct SolveJob {
  const uint64_t* masks;
  const float* y;
  const float* fef;
  float* phi;
  int32_t* info;
  const gnnshap_class* cls;  // device copy
  int64_t ncls, M, wpr, half, rb0, kr, nrb, ld, nch;
  double alpha, wr;
  uint64_t* T;
  int32_t* counts;
  double* dz;
  double* part;
  int64_t* usum;
  double* dv;
  double* scal;
  float* Wd;
  float* rv;                 // M: right-hand side, then z, then psi (panel path)
  int32_t panel;             // 1: the panel path, 0: one workgroup
  int32_t counts_in;         // 1: G~ is built from the counts as the panel path first reads each block
  int64_t tr0;               // first transpose item (64 rows x 64 players) of the job in the batch
};
// A system of the multi-block Cholesky path (more players than one
// workgroup takes, up to the iterative threshold) in a batch: the batched
// factorisation and triangular solves run every such system's steps in one
// launch each (one system per blockIdx.y).
struct MbJob {
  float* G;             // M x M, row stride ld: G~, then its Cholesky factor (lower)
  float* Winv;          // the inverse of the current 128-wide diagonal block
  float* rhs;           // M: the centred right-hand side, then L^-T x
  float* x;             // M
  const double* scal;   // the system's scalars (Delta at [3])
  float* phi;           // M
  int32_t* info;
  int64_t ld, M;
};

class CgGroup;
// gnnshap_solve_wls up to the iteration of an iterative system, which joins
// *grp (a group on `stream`, not full: the caller steps it); other systems
// are queued in full and grp is left as it was.  set_up_only (systems of the
// multi-block path): only the steps before the factorisation are queued; the
// caller runs the rest through launch_solve_mb.
int solve_wls_start(const gnnshap_sample_plan* plan, const gnnshap_class* classes, const uint64_t* masks,
                    const float* y, const float* f_empty_full, float* phi, int32_t* info, void* ws, size_t ws_bytes,
                    void* stream, CgGroup* grp, bool set_up_only = false);
// Whether a plan's system takes the multi-block Cholesky path, and its job
// (G, Winv, rhs, x, scal, ld, M from the workspace slice; the caller sets phi, info).
bool solve_multiblock(const gnnshap_sample_plan* plan);
int solve_fill_mb_job(const gnnshap_sample_plan* plan, const gnnshap_class* classes, void* slice, MbJob* job);
// The factorisation, both triangular solves and phi of n multi-block systems
// whose set-up has completed on `s` (max_M: their largest M).
int launch_solve_mb(const MbJob* jobs, int64_t n, int64_t max_M, hipStream_t s);
// Whether a plan's system is solved by one workgroup, the bytes of its slice, and the job fields it fixes.
bool solve_batchable(const gnnshap_sample_plan* plan);
size_t solve_slice_bytes(const gnnshap_sample_plan* plan);
int solve_fill_job(const gnnshap_sample_plan* plan, const gnnshap_class* classes, void* slice, SolveJob* job);
// The solve of a batch in launch sequences: the integer counts, their row
// sums and the scalars of G~ from the masks alone (they may run while the
// coalitions are evaluated), the right-hand side from the values, then G~
// and the factorisations.
int launch_solve_matrix(const SolveJob* jobs, int64_t n, int64_t max_M, int64_t max_wpr, int64_t max_nrb,
                        int64_t n_items, hipStream_t s);
// G~ in place of the counts for the jobs that do not build it as they read it
// (after launch_solve_matrix).
int launch_solve_build(const SolveJob* jobs, int64_t n, int64_t max_M, hipStream_t s);
int launch_solve_rhs(const SolveJob* jobs, int64_t n, int64_t max_M, int64_t max_wpr, int64_t max_half,
                     int64_t max_nch, hipStream_t s);
// Panel-path systems (J.panel): the factorisation of G~ (max_panels = the
// most 64-player panels of a job), which does not read the right-hand side,
// and the solve (centring, forward and backward substitution).  Other jobs
// are skipped by both.
int launch_panel_factor(const SolveJob* jobs, int64_t n, int64_t max_panels, hipStream_t s);
int launch_panel_solve(const SolveJob* jobs, int64_t n, hipStream_t s);
// The one-workgroup systems (factorisation and solves in one kernel; panel
// jobs are skipped).
int launch_solve_one(const SolveJob* jobs, int64_t n, hipStream_t s);
// Whether a one-workgroup-size system takes the panel path.
bool solve_panel_path(const gnnshap_sample_plan* plan);

}  // namespace gnnshap
