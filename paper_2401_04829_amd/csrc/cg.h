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
  int64_t* sitem;     // nsi: pass-A work items over the sparse rows, (first row << 8) | log2(lanes per row)
  int32_t* segcnt;    // 8 x max(rs, M): per-segment list lengths while the lists are built
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
  int64_t nsi;             // pass A's work items over the sparse rows (64 / lanes-per-row rows each)
  int32_t lgb;             // pass B: log2 of the lanes per player list (64 / 2^lgb players per wavefront)
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

// Several iterative solves advanced together on one stream.  Every chunk of
// iterations is one launch per pass for all members (one flat grid over the
// members' workgroups), so the members share the GPU inside each launch and
// the short passes of all members cost one launch latency instead of one
// each.  add() queues a new member's set-up on the stream (at most
// kCgGroupMax members at once); step() first waits for the chunk before the
// last one queued and reads the members' stop flags, queues phi and info of
// every member that has stopped and releases it, then queues the next chunk
// of iterations for the members left (each at its own iteration count), so
// at most two chunks are in flight; ready() says whether step() would return
// without waiting on the device.  Once empty() every member's phi and info
// are queued on the stream.  Each member holds a mapped stop flag; at most
// 16 are held per host thread at once.
constexpr int kCgGroupMax = 6;

class CgGroup {
 public:
  CgGroup();
  ~CgGroup();
  CgGroup(const CgGroup&) = delete;
  CgGroup& operator=(const CgGroup&) = delete;
  void set_stream(hipStream_t s) { s_ = s; }
  hipStream_t stream() const { return s_; }
  int add(const CgProblem& pr, const CgShape& sh, const CgWs& w);
  int size() const;
  bool empty() const { return size() == 0; }
  bool full() const { return size() >= kCgGroupMax; }
  bool ready() const;
  int step();
  // iterations of the member released last (-1 before any)
  int64_t last_iters() const { return last_iters_; }

 private:
  struct State;
  std::unique_ptr<State> st_;
  hipStream_t s_ = nullptr;
  int64_t last_iters_ = -1;
};

// Conjugate gradients on 1-perp for one system; returns once its phi and
// info are queued on `s` (the host waits on the stream for the stopping
// test).  *iters_out (may be null) receives the iterations run.
int cg_solve(const CgProblem& pr, const CgShape& sh, const CgWs& w, hipStream_t s, int64_t* iters_out);

// Largest number of players a plan's system is solved by factorisation for;
// larger systems are solved iteratively (Sec. 3.5 switches at 5000, the
// default when the plan's field is 0 or negative).
inline int64_t iterative_threshold(const gnnshap_sample_plan* p) {
  return p->iterative_threshold > 0 ? p->iterative_threshold : 5000;
}

}  // namespace gnnshap
