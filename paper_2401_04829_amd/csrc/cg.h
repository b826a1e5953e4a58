// Matrix-free solver of the projected Kernel-SHAP normal equations (Sec. 3.5:
// large systems are fitted iteratively instead of being factored).
#pragma once

#include <memory>

#include "common.h"

namespace gnnshap {

// Device state of one iterative solve.
struct CgState {
  double rr0;      // squared norm of the initial residual
  int32_t done;    // set by the iteration that stops
  int32_t iters;   // iterations run
  int32_t status;  // 0 converged, 1 iteration limit, 2 lost positive curvature
  int32_t pad;
};

// Buffers of the iterative solver, carved from the solve workspace.
struct CgWs {
  double* x;       // M: psi
  double* r;       // words_per_row * 64: residual, zero beyond M
  double* p;       // M: search direction
  double* s;       // M: A p
  double* upart;   // npc x kr: partial products R r per player chunk
  double* u;       // nrb * 64: R r, zero beyond kr
  double* qpart;   // nrc x M: partial products R^T u per row chunk
  double* uu;      // nbu x 2: partial |u|^2 and |m|.u
  double* usp;     // nsa x 2: the same over the sparse rows, per pass-A workgroup
  double* rr;      // 3 x nbc: partial r.r of iterations t mod 3
  double* hist;    // 2: step lengths of even and odd iterations
  int32_t* sz;     // kr: sizes of the random representative rows
  uint64_t* blocked;  // nrb x words_per_row x 64: the random rows in row blocks
  CgState* st;
  // sparse rows (random rows [0, rs), the smallest coalitions): their players
  int64_t* csr_ptr;   // rs + 1: players of each sparse row, ascending
  int32_t* csr_idx;   // nnz
  int64_t* csc_ptr;   // M + 1: rows of each player, ascending
  int32_t* csc_row;   // nnz
  double* qs;         // M: R_s^T u
};

// Launch shape of the iterative solver for M players and kr random
// representative rows (words_per_row mask words per row).
struct CgShape {
  int64_t M, wpr, kr, nrb;
  int64_t rs, nnz;         // sparse rows [0, rs) (whole row blocks), their players
  int64_t rbd0;            // first row block of the bit products (rs / 64)
  int64_t npc, pwords;     // product R r: player chunks of pwords words
  int64_t nrc, rbc;        // product R^T u: row chunks of rbc row blocks
  int64_t nbu, nbc;        // partial sums of the row pass (the sparse rows' total, then one per
                           // workgroup of bit rows; also its workgroups), workgroups of the player passes
  int64_t nsa, nsb;        // sparse workgroups of pass A (rows) and pass B (players)
  int64_t nrcd;            // row chunks of pass B's bit rows (0 without bit rows)
};
// The split of the random rows [rb0, rb0 + kr) of a class table into sparse
// rows (coalition size at most M / kSparseDiv, whole blocks of 64 rows) and
// bit rows; the shape of the solver for that split.
CgShape cg_shape(int64_t M, int64_t wpr, int64_t kr, int64_t rb0, const gnnshap_class* classes, int64_t ncls);
CgWs cg_carve(Carver& c, const CgShape& sh);

// The problem handed over by the solve entry point: the bit-transposed random
// rows T (nrb x M), the same rows in row blocks (word w of the 64 rows of
// block rb contiguous, rows beyond kr zero),
// the summed right-hand side dv (M, before centring) with its per-block sums
// bsum (nb of them), the class table (device) and the enumerated part alpha.
struct CgProblem {
  const uint64_t* T;
  const uint64_t* blocked;
  const double* dv;
  const double* bsum;
  int64_t nb;
  const gnnshap_class* classes;
  int64_t ncls;
  int64_t rb0;          // first random representative row
  double alpha;         // enumerated classes: their projected Gram is alpha P
  double wr;            // weight of every random row
  const float* fef;     // f(empty), f(full)
  float* phi;
  int32_t* info;
};

struct CgArgs;

// One iterative solve driven chunk by chunk, so that a caller can keep
// several solves in flight, each on its own stream: begin() queues the
// set-up; every step() first waits for the chunk before the last one queued
// and reads the stop flag it left, then (unless the iteration has stopped:
// done()) queues the next chunk of iterations, so at most two chunks are in
// flight; finish() waits for the last chunk, queues phi and info and leaves
// the object ready for another solve.  ready() says whether the next step()
// or finish() would return without waiting on the device, so one host
// thread can drive several solves by polling.  At most 8 solves per host
// thread are in flight at once (each holds a mapped stop flag).
class CgRun {
 public:
  CgRun();
  ~CgRun();
  CgRun(const CgRun&) = delete;
  CgRun& operator=(const CgRun&) = delete;
  int begin(const CgProblem& pr, const CgShape& sh, const CgWs& w, hipStream_t s);
  int step();
  bool done() const { return stopped_; }
  bool begun() const { return static_cast<bool>(st_); }
  bool ready() const;
  int finish(int64_t* iters_out);

 private:
  std::unique_ptr<CgArgs> st_;
  bool stopped_ = true;
};

// Conjugate gradients on 1-perp; returns once the iteration has stopped
// (the host waits on the stream for the stopping test) and phi/info are
// queued on `s`.  *iters_out (may be null) receives the iterations run.
int cg_solve(const CgProblem& pr, const CgShape& sh, const CgWs& w, hipStream_t s, int64_t* iters_out);

// Largest number of players a plan's system is solved by factorisation for;
// larger systems are solved iteratively (Sec. 3.5 switches at 5000, the
// default when the plan's field is 0 or negative).
inline int64_t iterative_threshold(const gnnshap_sample_plan* p) {
  return p->iterative_threshold > 0 ? p->iterative_threshold : 5000;
}

}  // namespace gnnshap
