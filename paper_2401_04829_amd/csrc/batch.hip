// Many targets per launch sequence: sampling, evaluation and the least squares
// of n explanations (Alg. 1 steps 2-5 of the GNNShap paper for each target),
// one launch per step for the whole batch, so small targets fill the GPU
// together instead of one after another.  Targets whose evaluation or system
// does not fit the batched kernels go through the single-target calls inside
// the same sequence; every value is the one the single-target calls give.
#include <algorithm>
#include <atomic>
#include <chrono>
#include <condition_variable>
#include <cstring>
#include <functional>
#include <mutex>
#include <thread>
#include <vector>

#include "batch.h"
#include "cg.h"
#include "common.h"

namespace gnnshap {

// Side streams of the current device for the calling thread, each with the
// events that fork work onto it and join it back, and one more (created on first use,
// default priority, kept until the process ends).  Two: with the caller's
// stream and the extraction stream of a pipelined caller that makes four,
// the number of hardware queues a process gets by default, so no two of them
// share a queue.
constexpr int kSideStreams = 2;

struct SideStream {
  hipStream_t stream = nullptr;
  hipEvent_t fork = nullptr, join = nullptr, aux = nullptr;
  hipEvent_t rest_out = nullptr;   // end of the one-by-one solves queued on this stream
};

struct DeviceSides {
  int device = -1;
  SideStream side[kSideStreams];
};

SideStream* side_stream(int i) {
  static thread_local std::vector<DeviceSides> per_device;
  int dev = 0;
  if (i < 0 || i >= kSideStreams || hipGetDevice(&dev) != hipSuccess) return nullptr;
  for (DeviceSides& d : per_device)
    if (d.device == dev) return &d.side[i];
  DeviceSides d;
  d.device = dev;
  for (SideStream& x : d.side) {
    if (hipStreamCreateWithFlags(&x.stream, hipStreamNonBlocking) != hipSuccess ||
        hipEventCreateWithFlags(&x.fork, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&x.join, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&x.aux, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&x.rest_out, hipEventDisableTiming) != hipSuccess) {
      (void)hipGetLastError();
      return nullptr;
    }
  }
  per_device.push_back(d);
  return &per_device.back().side[i];
}

// A host thread that issues one target group's launches while the calling
// thread issues the other's: every launch and event costs a few
// microseconds of host time, and for a batch of 100 small targets that host
// time, not the GPU, bounds the step.  One per calling thread, created on
// first use; between jobs it spins for up to kSpinUs, then sleeps.
class Issuer {
 public:
  static constexpr int kSpinUs = 1000;
  Issuer() : th_([this] { loop(); }) {}
  ~Issuer() {
    {
      std::lock_guard<std::mutex> lk(mu_);
      stop_ = true;
    }
    cv_.notify_one();
    th_.join();
  }
  // Runs f on the worker (with `device` current) and returns at once.
  void post(int device, std::function<int()> f) {
    {
      std::lock_guard<std::mutex> lk(mu_);
      job_ = std::move(f);
      device_ = device;
      state_.store(1, std::memory_order_release);
    }
    cv_.notify_one();
  }
  // Waits for the posted job; its status, with its error text copied to the
  // calling thread.
  int wait() {
    while (state_.load(std::memory_order_acquire) != 2) std::this_thread::yield();
    state_.store(0, std::memory_order_relaxed);
    if (status_ != GNNSHAP_OK) return fail(status_, "%s", msg_);
    return GNNSHAP_OK;
  }

 private:
  void loop() {
    for (;;) {
      const auto t0 = std::chrono::steady_clock::now();
      while (state_.load(std::memory_order_acquire) != 1 &&
             std::chrono::steady_clock::now() - t0 < std::chrono::microseconds(kSpinUs))
        std::this_thread::yield();
      std::function<int()> f;
      int dev = 0;
      {
        std::unique_lock<std::mutex> lk(mu_);
        cv_.wait(lk, [this] { return stop_ || state_.load(std::memory_order_acquire) == 1; });
        if (stop_) return;
        f = std::move(job_);
        dev = device_;
      }
      int st = hipSetDevice(dev) == hipSuccess ? GNNSHAP_OK : fail(GNNSHAP_EHIP, "hipSetDevice failed");
      if (st == GNNSHAP_OK) st = f();
      status_ = st;
      std::strncpy(msg_, st == GNNSHAP_OK ? "" : gnnshap_last_error(), sizeof(msg_) - 1);
      msg_[sizeof(msg_) - 1] = 0;
      state_.store(2, std::memory_order_release);
    }
  }
  std::mutex mu_;
  std::condition_variable cv_;
  std::function<int()> job_;
  int device_ = 0;
  std::atomic<int> state_{0};      // 0 idle, 1 posted, 2 done
  int status_ = GNNSHAP_OK;
  char msg_[512] = "";
  bool stop_ = false;
  std::thread th_;
};

Issuer& issuer() {
  static thread_local Issuer w;
  return w;
}

// At least n events of the calling thread (created on demand, default flags
// without timing, kept until the process ends), or nullptr.
hipEvent_t* event_pool(size_t n) {
  static thread_local std::vector<hipEvent_t> pool;
  while (pool.size() < n) {
    hipEvent_t e = nullptr;
    if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) {
      (void)hipGetLastError();
      return nullptr;
    }
    pool.push_back(e);
  }
  return pool.data();
}

struct DeviceStages {
  int device = -1;
  HostStage ring[2][2];
  int next[2] = {0, 0};
};

HostStage* host_stage(size_t bytes, int ring) {
  static thread_local std::vector<DeviceStages> per_device;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return nullptr;
  DeviceStages* d = nullptr;
  for (DeviceStages& x : per_device)
    if (x.device == dev) d = &x;
  if (!d) {
    per_device.emplace_back();
    d = &per_device.back();
    d->device = dev;
  }
  if (ring < 0 || ring > 1) return nullptr;
  HostStage* h = &d->ring[ring][d->next[ring]];
  d->next[ring] ^= 1;
  // Growing a buffer (page-locked allocation takes milliseconds) grows the
  // other buffer of the ring too when it is idle, so that the cost falls on
  // one call.
  const size_t want = bytes + bytes / 2 + 4096;
  for (HostStage* x : {h, &d->ring[ring][d->next[ring]]}) {
    if (!x->done && hipEventCreateWithFlags(&x->done, hipEventDisableTiming) != hipSuccess) return nullptr;
    if (x != h && (x->pending || x->cap >= bytes)) continue;
    if (x->pending && hipEventSynchronize(x->done) != hipSuccess) return nullptr;
    x->pending = false;
    if (x->cap >= bytes) continue;
    if (x->buf) (void)hipHostFree(x->buf);
    x->buf = nullptr;
    x->cap = 0;
    void* p = nullptr;
    // coherent: the GPU reads it uncached, so a reused buffer is never stale
    if (hipHostMalloc(&p, want, hipHostMallocMapped | hipHostMallocCoherent) != hipSuccess) {
      (void)hipGetLastError();
      return nullptr;
    }
    x->buf = static_cast<char*>(p);
    x->cap = want;
  }
  return h;
}

__global__ void __launch_bounds__(256) k_copy16(const uint4* __restrict__ src, uint4* __restrict__ dst, size_t n) {
  for (size_t i = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x; i < n; i += static_cast<size_t>(gridDim.x) * 256)
    dst[i] = src[i];
}

int copy_by_kernel(void* dst, const void* src, size_t bytes, hipStream_t s) {
  const size_t n = (bytes + 15) / 16;
  if (n == 0) return GNNSHAP_OK;
  if ((reinterpret_cast<uintptr_t>(dst) | reinterpret_cast<uintptr_t>(src)) & 15)
    return fail(GNNSHAP_EINVAL, "copy buffers must be 16-byte aligned");
  k_copy16<<<grid_for(static_cast<int64_t>(n), 256, 256), 256, 0, s>>>(static_cast<const uint4*>(src),
                                                                       static_cast<uint4*>(dst), n);
  GS_HIP(hipGetLastError());
  return GNNSHAP_OK;
}

}  // namespace gnnshap

namespace {

struct Layout {
  int64_t n = 0, classes = 0;
  std::vector<int64_t> mask_off, row_off, player_off, class_off;
  std::vector<size_t> eval_bytes, solve_bytes;
};

// The model of a batch: a GCN (gcn) or a two-layer GAT (gat), exactly one set.
struct Model {
  const gnnshap_gcn* gcn = nullptr;
  const gnnshap_gat* gat = nullptr;
};

int make_layout(const gnnshap_subgraph* sgs, const gnnshap_sample_plan* plans, int64_t n, Model m, Layout* L) {
  if (!sgs || !plans || !(m.gcn || m.gat) || n < 1) return gnnshap::fail(GNNSHAP_EINVAL, "null argument or n < 1");
  if (n > 65535) return gnnshap::fail(GNNSHAP_EUNSUPPORTED, "at most 65535 targets per batch");
  L->n = n;
  L->mask_off.resize(n + 1);
  L->row_off.resize(n + 1);
  L->player_off.resize(n + 1);
  L->class_off.resize(n + 1);
  L->eval_bytes.resize(n);
  L->solve_bytes.resize(n);
  L->mask_off[0] = L->row_off[0] = L->player_off[0] = L->class_off[0] = 0;
  for (int64_t t = 0; t < n; ++t) {
    const gnnshap_sample_plan& p = plans[t];
    if (p.num_players != sgs[t].num_edges)
      return gnnshap::fail(GNNSHAP_EINVAL, "plan %lld is not for subgraph %lld's players", (long long)t, (long long)t);
    size_t eb = 0, sb = 0;
    if (int st = m.gcn ? gnnshap_eval_workspace(&sgs[t], m.gcn, p.num_rows, &eb)
                       : gnnshap_gat_eval_workspace(&sgs[t], m.gat, p.num_rows, &eb))
      return st;
    if (int st = gnnshap_solve_workspace(&p, &sb)) return st;
    L->eval_bytes[t] = eb;
    L->solve_bytes[t] = sb;
    L->mask_off[t + 1] = L->mask_off[t] + p.num_rows * p.words_per_row;
    L->row_off[t + 1] = L->row_off[t] + p.num_rows;
    L->player_off[t + 1] = L->player_off[t] + p.num_players;
    L->class_off[t + 1] = L->class_off[t] + p.num_classes;
  }
  L->classes = L->class_off[n];
  return GNNSHAP_OK;
}

struct BatchWs {
  gnnshap_class* classes;
  gnnshap::SampleJob* sample;
  gnnshap::EvalJob* eval;
  gnnshap::SolveJob* solve;
  gnnshap::MbJob* mb;
  std::vector<char*> eval_slice, solve_slice;
};

BatchWs carve(gnnshap::Carver& c, const Layout& L) {
  BatchWs b;
  b.classes = c.take<gnnshap_class>(L.classes);
  b.sample = c.take<gnnshap::SampleJob>(L.n);
  b.eval = c.take<gnnshap::EvalJob>(L.n);
  b.solve = c.take<gnnshap::SolveJob>(L.n);
  b.mb = c.take<gnnshap::MbJob>(L.n);
  b.eval_slice.resize(L.n);
  b.solve_slice.resize(L.n);
  for (int64_t t = 0; t < L.n; ++t) b.eval_slice[t] = c.take<char>(L.eval_bytes[t]);
  for (int64_t t = 0; t < L.n; ++t) b.solve_slice[t] = c.take<char>(L.solve_bytes[t]);
  return b;
}

// The target order (group 0 first, each group in target order) and the
// group boundaries: group g = order[bound[g], bound[g+1]).  Group 0 holds the
// systems that take the panel path, group 1 the rest; a batch with only one
// kind runs as one group.
void split_groups(const gnnshap_sample_plan* plans, int64_t n, std::vector<int64_t>* order, int64_t bound[3]) {
  order->clear();
  order->reserve(n);
  bound[0] = 0;
  for (int g = 0; g < 2; ++g) {
    for (int64_t t = 0; t < n; ++t)
      if ((gnnshap::solve_panel_path(&plans[t]) ? 0 : 1) == g) order->push_back(t);
    bound[g + 1] = static_cast<int64_t>(order->size());
  }
  if (bound[1] == n) bound[1] = 0;   // only panel-path systems: one group
}

}  // namespace

namespace {

int batch_workspace(const gnnshap_subgraph* sgs, const gnnshap_sample_plan* plans, int64_t n, Model m,
                    size_t* bytes) {
  gnnshap::clear_error();
  if (!bytes) return gnnshap::fail(GNNSHAP_EINVAL, "bytes is NULL");
  Layout L;
  if (int st = make_layout(sgs, plans, n, m, &L)) return st;
  gnnshap::Carver c(nullptr);
  carve(c, L);
  *bytes = c.bytes();
  return GNNSHAP_OK;
}

int explain_batch_impl(const gnnshap_subgraph* sgs, const gnnshap_sample_plan* plans, const gnnshap_class* classes,
                       int64_t n, Model mdl, const float* X, int32_t target_class, uint64_t* masks, float* weights,
                       float* y, float* f_empty_full, int32_t* class_out, float* phi, int32_t* info, void* ws,
                       size_t ws_bytes, void* stream) {
  GS_TRY_BEGIN
  gnnshap::clear_error();
  Layout L;
  if (int st = make_layout(sgs, plans, n, mdl, &L)) return st;
  const gnnshap_gcn* model = mdl.gcn;
  if (!classes || !masks || !weights || !y || !f_empty_full || !phi || !info || !ws)
    return gnnshap::fail(GNNSHAP_EINVAL, "null argument");
  gnnshap::Carver need(nullptr);
  carve(need, L);
  if (ws_bytes < need.bytes()) return gnnshap::fail(GNNSHAP_ECAPACITY, "batch workspace needs %zu bytes", need.bytes());
  gnnshap::Carver cv(ws);
  const BatchWs b = carve(cv, L);
  hipStream_t s = static_cast<hipStream_t>(stream);
  for (int64_t t = 0; t < n; ++t) {
    if (plans[t].num_players > 131072)
      return gnnshap::fail(GNNSHAP_EUNSUPPORTED, "sampler supports up to 131072 players");
    int64_t row = 0;
    const gnnshap_class* ct = classes + L.class_off[t];
    for (int64_t i = 0; i < plans[t].num_classes; ++i) {
      if (ct[i].row_begin != row || ct[i].row_count < 1 || ct[i].size < 1 ||
          2 * static_cast<int64_t>(ct[i].size) > plans[t].num_players)
        return gnnshap::fail(GNNSHAP_EINVAL, "class table of target %lld inconsistent", (long long)t);
      row += ct[i].row_count;
    }
    if (row != plans[t].num_rows / 2) return gnnshap::fail(GNNSHAP_EINVAL, "class table of target %lld short", (long long)t);
  }
  // Targets run in two groups when both kinds of systems are present: the
  // largest ones (panel path, whose factorisations set the length of the
  // whole sequence) and their sampling and evaluation on a side stream, the
  // rest on `stream`, each step launched for both groups before the next, so
  // that the long factorisations overlap the other group's work.
  std::vector<int64_t> order;
  int64_t bound[3];
  split_groups(plans, n, &order, bound);

  // The class tables and the four job tables (in group order) sit at the
  // front of the workspace; they are assembled in a host image of that range
  // and copied in one transfer before the first launch.
  char* const base = static_cast<char*>(ws);
  const size_t front = static_cast<size_t>(reinterpret_cast<char*>(b.mb + n) - base);
  gnnshap::HostStage* stage = gnnshap::host_stage(front, 0);
  if (!stage) return gnnshap::fail(GNNSHAP_EHIP, "page-locked staging allocation failed");
  char* const image = stage->buf;
  std::fill(image, image + front, 0);
  auto at = [&](const void* dev_ptr) { return image + (static_cast<const char*>(dev_ptr) - base); };
  std::copy(classes, classes + L.classes, reinterpret_cast<gnnshap_class*>(at(b.classes)));
  gnnshap::SampleJob* sj = reinterpret_cast<gnnshap::SampleJob*>(at(b.sample));
  gnnshap::EvalJob* ej = reinterpret_cast<gnnshap::EvalJob*>(at(b.eval));
  gnnshap::SolveJob* vj = reinterpret_cast<gnnshap::SolveJob*>(at(b.solve));
  gnnshap::MbJob* mj = reinterpret_cast<gnnshap::MbJob*>(at(b.mb));

  struct Group {
    int64_t begin = 0, end = 0;                      // range of order[]
    int64_t max_wpr = 0, max_k = 0;                  // sampling
    bool eval_all = false;                           // batched evaluation
    int64_t max_nodes = 0, max_ndst = 0, max_n1 = 0, rows_jobs = 0;
    size_t rows_lds = 0;
    int64_t solve_begin = 0, solve_count = 0;        // range of the solve job table
    int64_t bM = 0, bw = 0, bh = 0, bnrb = 0, bnch = 0;
    int64_t max_panels = 0;                          // of the panel-path systems
    bool small = false;                              // some one-workgroup system
    std::vector<int64_t> rest;                       // targets solved one by one
    std::vector<int64_t> mb;                         // of them, multi-block systems: their index in the MbJob table, else -1
  } grp[2];
  for (int g = 0; g < 2; ++g) {
    grp[g].begin = bound[g];
    grp[g].end = bound[g + 1];
  }
  int64_t nv = 0, nmb = 0;
  std::vector<int64_t> rest_pos(static_cast<size_t>(n), -1);   // index of a target in its group's rest list
  int64_t tr_items = 0;   // transpose items (64 rows x 64 players) of the batched systems
  for (Group& G : grp) {
    // 1. sampling jobs
    for (int64_t j = G.begin; j < G.end; ++j) {
      const int64_t t = order[j];
      const gnnshap_sample_plan& p = plans[t];
      sj[j] = gnnshap::SampleJob{b.classes + L.class_off[t], p.num_classes, p.num_rows / 2, p.num_players,
                                 p.words_per_row, static_cast<uint32_t>(p.seed), static_cast<uint32_t>(p.seed >> 32),
                                 static_cast<uint32_t>(p.stream_id), static_cast<uint32_t>(p.stream_id >> 32),
                                 masks + L.mask_off[t], weights + L.row_off[t]};
      G.max_wpr = std::max(G.max_wpr, p.words_per_row);
      G.max_k = std::max(G.max_k, p.num_rows);
    }
    // 2. coalition-value jobs (two-layer models with X W_1 given)
    G.eval_all = model && model->num_layers == 2 && model->XW1;
    for (int64_t j = G.begin; j < G.end && G.eval_all; ++j)
      G.eval_all = gnnshap::eval_batchable(&sgs[order[j]], model, plans[order[j]].num_rows);
    if (G.eval_all) {
      for (int64_t j = G.begin; j < G.end; ++j) {
        const int64_t t = order[j];
        const gnnshap_subgraph& g = sgs[t];
        gnnshap::EvalJob& J = ej[j];
        J = gnnshap::EvalJob{};
        J.node_gid = g.node_gid;
        J.dst_ptr = g.dst_ptr;
        J.edge_src = g.edge_src;
        J.n_nodes = g.num_nodes;
        J.n_dst = g.num_dst;
        J.n1 = g.hop_ptr[2];
        J.M = g.num_edges;
        J.wpr = plans[t].words_per_row;
        J.k = plans[t].num_rows;
        J.masks = masks + L.mask_off[t];
        J.y = y + L.row_off[t];
        J.fef = f_empty_full + 2 * t;
        J.cls_out = class_out ? class_out + t : nullptr;
        gnnshap::eval_carve_slice(b.eval_slice[t], &g, model, J.k, &J);
        const size_t rl = gnnshap::eval_rows_lds(&g, model);
        J.rows_ok = rl > 0 ? 1 : 0;
        G.rows_jobs += J.rows_ok;
        G.rows_lds = std::max(G.rows_lds, rl);
        G.max_nodes = std::max(G.max_nodes, J.n_nodes);
        G.max_ndst = std::max(G.max_ndst, J.n_dst);
        G.max_n1 = std::max(G.max_n1, J.n1);
      }
    }
    // 3. least-squares jobs: one-workgroup systems batched, the rest one by one
    G.solve_begin = nv;
    for (int64_t j = G.begin; j < G.end; ++j) {
      const int64_t t = order[j];
      const gnnshap_sample_plan& p = plans[t];
      if (!gnnshap::solve_batchable(&p)) {
        rest_pos[t] = static_cast<int64_t>(G.rest.size());
        G.rest.push_back(t);
        int64_t m = -1;
        if (gnnshap::solve_multiblock(&p)) {
          gnnshap::MbJob& J = mj[nmb];
          if (int st = gnnshap::solve_fill_mb_job(&p, classes + L.class_off[t], b.solve_slice[t], &J)) return st;
          J.phi = phi + L.player_off[t];
          J.info = info + t;
          m = nmb++;
        }
        G.mb.push_back(m);
        continue;
      }
      gnnshap::SolveJob J{};
      if (int st = gnnshap::solve_fill_job(&p, classes + L.class_off[t], b.solve_slice[t], &J)) return st;
      J.masks = masks + L.mask_off[t];
      J.y = y + L.row_off[t];
      J.fef = f_empty_full + 2 * t;
      J.phi = phi + L.player_off[t];
      J.info = info + t;
      J.cls = b.classes + L.class_off[t];
      J.tr0 = tr_items;
      if (J.kr > 0) tr_items += J.nrb * J.wpr;
      G.bM = std::max(G.bM, J.M);
      G.bw = std::max(G.bw, J.wpr);
      G.bh = std::max(G.bh, J.half);
      G.bnrb = std::max(G.bnrb, J.nrb);
      G.bnch = std::max(G.bnch, J.nch);
      if (gnnshap::solve_panel_path(&p)) G.max_panels = std::max(G.max_panels, gnnshap::ceil_div(J.M, 64));
      else G.small = true;
      vj[nv++] = J;
    }
    G.solve_count = nv - G.solve_begin;
  }

  // one sampling launch for the whole batch
  const int64_t sample_blocks = gnnshap::plan_sample_batch(sj, n);
  const int64_t sample_wpr = std::max(grp[0].max_wpr, grp[1].max_wpr);
  // one G~ pass for every batched system
  int64_t mM = 0, mw = 0, mnrb = 0;
  for (const Group& G : grp) {
    mM = std::max(mM, G.bM);
    mw = std::max(mw, G.bw);
    mnrb = std::max(mnrb, G.bnrb);
  }

  if (int st = gnnshap::copy_by_kernel(ws, image, front, s)) return st;
  GS_HIP(hipEventRecord(stage->done, s));
  stage->pending = true;
  // Every launch after the job-table copy, on origin stream `o` and the side
  // streams forked from it.
  auto issue = [&](hipStream_t o) -> int {
      // Streams: the masks of every target are sampled on origin stream `o`;
      // then group 0 (the panel-path systems) is evaluated and solved on side
      // stream 0, group 1 on `o`, and G~ of every batched system is built on
      // side stream 1 while the coalitions are evaluated.  Three event pairs:
      // the fork after sampling (side streams 0 and 1 wait on it), G~ ready
      // (both factorisations wait on it) and the join of side stream 0.  The
      // launches of side stream 0 are issued by the worker thread while this
      // thread issues the others.
      gnnshap::SideStream* side0 = nullptr;
      gnnshap::SideStream* mat = nullptr;
      if (grp[0].end > grp[0].begin) {
        side0 = gnnshap::side_stream(0);
        if (!side0) return gnnshap::fail(GNNSHAP_EHIP, "could not create a side stream");
      }
      if (nv > 0) {
        mat = gnnshap::side_stream(1);
        if (!mat) return gnnshap::fail(GNNSHAP_EHIP, "could not create a side stream");
      }
      hipStream_t gs[2] = {side0 ? side0->stream : o, o};
      if (int st = gnnshap::launch_sample_batch(b.sample, n, sample_blocks, sample_wpr, o)) return st;
      if (side0 || mat) {
        gnnshap::SideStream* f = side0 ? side0 : mat;
        GS_HIP(hipEventRecord(f->fork, o));
        if (side0) GS_HIP(hipStreamWaitEvent(side0->stream, f->fork, 0));
        if (mat) GS_HIP(hipStreamWaitEvent(mat->stream, f->fork, 0));
      }
      hipEvent_t* ev_pool = gnnshap::event_pool(static_cast<size_t>(n));
      if (!ev_pool) return gnnshap::fail(GNNSHAP_EHIP, "could not create events");
      std::vector<hipEvent_t> evaluated(static_cast<size_t>(n), nullptr);
      // The systems solved one by one (too large for the batched kernels).
      // The factored ones are queued as soon as their values are queued (from
      // eval_group, target by target), in turn on the two side streams, so
      // that they run beside the evaluation of later targets: a
      // one-workgroup system in full; the multi-block systems in runs of
      // kMbRun, each run's set-ups on one stream followed by one batched
      // factorisation and solve of the whole run (launch_solve_mb: one launch
      // per step for all of them instead of one per system).  The iterative
      // ones go to two solver groups, one on each side stream, each holding up
      // to kPerGroup systems: a group takes a system once its values are there
      // (a host query of its evaluation event, so a side stream never waits
      // for a later target) and advances its systems together; the host steps
      // whichever group can move without waiting.  Two groups let one group's
      // short passes and launch tails overlap the other's long passes.  Both
      // side streams are joined back into `home` at the end.  A single system
      // runs on `home`.
      struct Rest {
        hipStream_t home = nullptr;
        gnnshap::SideStream* side[2] = {nullptr, nullptr};
        gnnshap::CgGroup cg[2];
        gnnshap::CgGroup on_home;     // stays empty: factored systems are queued in full
        int ng = 0;                   // solver groups (0: not opened)
        int turn = 0;                 // carrier of the next factored system or run
        int64_t run_begin = -1, run_n = 0, run_M = 0;   // the open run of multi-block systems
        size_t taken = 0;             // rest[0, taken) queued or listed in its
        std::vector<int64_t> its;     // iterative systems, in order
      };
      Rest rst[2];
      constexpr int kPerGroup = 3;
      constexpr int64_t kMbRun = 24;
      auto rest_open = [&](int gi, hipStream_t home) -> int {
        Rest& R = rst[gi];
        const std::vector<int64_t>& rest = grp[gi].rest;
        R.home = home;
        R.on_home.set_stream(home);
        R.ng = 1;
        R.cg[0].set_stream(home);
        if (rest.size() >= 2) {
          for (int i = 0; i < 2; ++i) {
            R.side[i] = gnnshap::side_stream(i);
            if (!R.side[i]) return gnnshap::fail(GNNSHAP_EHIP, "could not create a side stream");
            R.cg[i].set_stream(R.side[i]->stream);
          }
          R.ng = 2;
        }
        return GNNSHAP_OK;
      };
      auto rest_start = [&](Rest& R, int64_t t, gnnshap::CgGroup* g, bool set_up_only) -> int {
        const hipStream_t st = g->stream();
        if (st != R.home) {
          // the target's values (and through them its masks) are ready
          if (!evaluated[t]) return gnnshap::fail(GNNSHAP_EHIP, "target %lld has no evaluation event",
                                                  static_cast<long long>(t));
          GS_HIP(hipStreamWaitEvent(st, evaluated[t], 0));
        }
        return gnnshap::solve_wls_start(&plans[t], classes + L.class_off[t], masks + L.mask_off[t], y + L.row_off[t],
                                        f_empty_full + 2 * t, phi + L.player_off[t], info + t, b.solve_slice[t],
                                        L.solve_bytes[t], st, g, set_up_only);
      };
      // a factored system only takes its carrier's stream (no member is added)
      auto carrier = [&](Rest& R) -> gnnshap::CgGroup* { return R.ng == 2 ? &R.cg[R.turn] : &R.on_home; };
      auto close_run = [&](Rest& R) -> int {
        if (R.run_n == 0) return GNNSHAP_OK;
        if (int st = gnnshap::launch_solve_mb(b.mb + R.run_begin, R.run_n, R.run_M, carrier(R)->stream())) return st;
        R.run_n = 0;
        R.run_M = 0;
        R.turn ^= R.ng == 2 ? 1 : 0;
        return GNNSHAP_OK;
      };
      // queue the factored systems of rest[taken, upto) (their values are queued)
      auto rest_take = [&](int gi, size_t upto) -> int {
        Rest& R = rst[gi];
        const Group& Gr = grp[gi];
        for (; R.taken < upto; ++R.taken) {
          const size_t i = R.taken;
          const int64_t t = Gr.rest[i];
          if (plans[t].num_players > gnnshap::iterative_threshold(&plans[t])) {
            R.its.push_back(t);
          } else if (Gr.mb[i] >= 0) {
            if (R.run_n == 0) R.run_begin = Gr.mb[i];
            if (int st = rest_start(R, t, carrier(R), true)) return st;
            R.run_M = std::max<int64_t>(R.run_M, plans[t].num_players);
            if (++R.run_n == kMbRun)
              if (int st = close_run(R)) return st;
          } else {
            if (int st = rest_start(R, t, carrier(R), false)) return st;
            if (R.run_n == 0) R.turn ^= R.ng == 2 ? 1 : 0;
          }
        }
        return GNNSHAP_OK;
      };
      auto rest_finish = [&](int gi) -> int {
        Rest& R = rst[gi];
        if (grp[gi].rest.empty()) return GNNSHAP_OK;
        if (int st = rest_take(gi, grp[gi].rest.size())) return st;
        if (int st = close_run(R)) return st;
        auto evaluated_done = [&](int64_t t) {
          const hipError_t q = hipEventQuery(evaluated[t]);
          if (q == hipErrorNotReady) {
            (void)hipGetLastError();
            return false;
          }
          return true;   // complete, or an error that the stream wait reports
        };
        const int ng = R.ng;
        const int cap = ng == 1 ? gnnshap::kCgGroupMax : kPerGroup;
        size_t next = 0;
        for (;;) {
          bool moved = false, busy = false;
          while (next < R.its.size()) {
            int gi2 = -1;
            for (int i = 0; i < ng; ++i)
              if (R.cg[i].size() < cap && (gi2 < 0 || R.cg[i].size() < R.cg[gi2].size())) gi2 = i;
            if (gi2 < 0) break;
            const int64_t t = R.its[next];
            if (R.cg[gi2].stream() != R.home && evaluated[t] && !evaluated_done(t)) break;
            if (int st = rest_start(R, t, &R.cg[gi2], false)) return st;
            ++next;
            moved = true;
          }
          for (int i = 0; i < ng; ++i) {
            if (R.cg[i].empty()) continue;
            busy = true;
            if (!R.cg[i].ready()) continue;
            if (int st = R.cg[i].step()) return st;
            moved = true;
          }
          if (!busy && next >= R.its.size()) break;
          if (!moved) std::this_thread::sleep_for(std::chrono::microseconds(20));
        }
        for (int i = 0; i < 2; ++i) {
          if (!R.side[i]) continue;
          GS_HIP(hipEventRecord(R.side[i]->rest_out, R.side[i]->stream));
          GS_HIP(hipStreamWaitEvent(R.home, R.side[i]->rest_out, 0));
        }
        return GNNSHAP_OK;
      };
      // coalition values of group gi; evaluated[t] is an event recorded on the
      // group's stream once target t's values are there (so that its solve
      // can start on another stream while later targets are evaluated, and
      // is queued right away)
      auto eval_group = [&](int gi) -> int {
        const Group& G = grp[gi];
        if (G.end == G.begin) return GNNSHAP_OK;
        int st_eval = GNNSHAP_EUNSUPPORTED;
        if (G.eval_all) {
          const gnnshap::EvalModel md{model->XW1, model->b ? model->b[0] : nullptr, model->W[1],
                                      model->b ? model->b[1] : nullptr, model->dims[1], model->dims[2], target_class};
          st_eval = gnnshap::launch_eval_batch(b.eval + G.begin, G.end - G.begin, md, G.max_nodes, G.max_ndst, G.max_n1,
                                               G.max_wpr, G.max_k, G.rows_jobs, G.rows_lds, gs[gi]);
          if (st_eval != GNNSHAP_OK && st_eval != GNNSHAP_EUNSUPPORTED) return st_eval;
          gnnshap::clear_error();
          if (st_eval == GNNSHAP_OK) {
            GS_HIP(hipEventRecord(ev_pool[G.begin], gs[gi]));
            for (int64_t j = G.begin; j < G.end; ++j) evaluated[order[j]] = ev_pool[G.begin];
          }
        }
        if (st_eval != GNNSHAP_OK) {
          for (int64_t j = G.begin; j < G.end; ++j) {
            const int64_t t = order[j];
            const gnnshap_sample_plan& p = plans[t];
            if (model) {
              if (int st = gnnshap::eval_coalitions_impl(&sgs[t], model, X, target_class, masks + L.mask_off[t],
                                                         p.num_rows, p.words_per_row, y + L.row_off[t],
                                                         f_empty_full + 2 * t, class_out ? class_out + t : nullptr,
                                                         b.eval_slice[t], L.eval_bytes[t], gs[gi], true))
                return st;
            } else if (int st = gnnshap_gat_eval_coalitions(&sgs[t], mdl.gat, target_class, masks + L.mask_off[t],
                                                            p.num_rows, p.words_per_row, y + L.row_off[t],
                                                            f_empty_full + 2 * t, class_out ? class_out + t : nullptr,
                                                            b.eval_slice[t], L.eval_bytes[t], gs[gi])) {
              return st;
            }
            GS_HIP(hipEventRecord(ev_pool[j], gs[gi]));
            evaluated[t] = ev_pool[j];
            if (rest_pos[t] >= 0)
              if (int st = rest_take(gi, static_cast<size_t>(rest_pos[t]) + 1)) return st;
          }
        }
        return GNNSHAP_OK;
      };
      // right-hand side, then the factorisations and solves of group gi:
      // one-workgroup systems (G~ built in place, then factorisation and
      // solves in one kernel) once the counts are ready; panel-path systems
      // factored on the matrix stream right behind the counts (building G~ as
      // each block is first read; the factorisation does not read the
      // right-hand side), then solved on the group's stream once both are ready
      auto solve_group = [&](int gi) -> int {
        const Group& G = grp[gi];
        if (G.solve_count > 0) {
          const gnnshap::SolveJob* jb = b.solve + G.solve_begin;
          if (int st = gnnshap::launch_solve_rhs(jb, G.solve_count, G.bM, G.bw, G.bh, G.bnch, gs[gi])) return st;
          if (G.max_panels > 0) {
            if (int st = gnnshap::launch_panel_factor(jb, G.solve_count, G.max_panels, mat->stream)) return st;
            GS_HIP(hipEventRecord(mat->aux, mat->stream));
            GS_HIP(hipStreamWaitEvent(gs[gi], mat->aux, 0));
            if (int st = gnnshap::launch_panel_solve(jb, G.solve_count, gs[gi])) return st;
          }
          if (G.small) {
            GS_HIP(hipStreamWaitEvent(gs[gi], mat->join, 0));
            if (int st = gnnshap::launch_solve_build(jb, G.solve_count, G.bM, gs[gi])) return st;
            if (int st = gnnshap::launch_solve_one(jb, G.solve_count, gs[gi])) return st;
          }
        }
        return rest_finish(gi);
      };
      // G~ first: it depends on the masks only, and queued ahead of the
      // evaluations it gets the GPU before their many workgroups fill it
      int st = GNNSHAP_OK;
      if (mat) {
        st = gnnshap::launch_solve_matrix(b.solve, nv, mM, mw, mnrb, tr_items, mat->stream);
        if (st == GNNSHAP_OK && hipEventRecord(mat->join, mat->stream) != hipSuccess)
          st = gnnshap::fail(GNNSHAP_EHIP, "hipEventRecord failed");
        if (st != GNNSHAP_OK) return st;
      }
      // group 0 on the worker: evaluation, right-hand side, factorisation, join record
      gnnshap::Issuer* worker = nullptr;
      if (side0) {
        int dev = 0;
        GS_HIP(hipGetDevice(&dev));
        worker = &gnnshap::issuer();
        worker->post(dev, [&]() -> int {
          if (int st = rest_open(0, gs[0])) return st;
          if (int st = eval_group(0)) return st;
          if (int st = solve_group(0)) return st;
          GS_HIP(hipEventRecord(side0->join, side0->stream));
          return GNNSHAP_OK;
        });
      }
      st = rest_open(1, gs[1]);
      if (st == GNNSHAP_OK) st = eval_group(1);
      if (st == GNNSHAP_OK) st = solve_group(1);
      if (worker) {
        const int wst = worker->wait();
        if (st == GNNSHAP_OK) st = wst;
        if (st == GNNSHAP_OK && hipStreamWaitEvent(o, side0->join, 0) != hipSuccess)
          st = gnnshap::fail(GNNSHAP_EHIP, "hipStreamWaitEvent failed");
      }
      return st;
  };
  if (int st = issue(s)) return st;
  return GNNSHAP_OK;
  GS_TRY_END
}

}  // namespace

extern "C" int gnnshap_explain_batch_workspace(const gnnshap_subgraph* sgs, const gnnshap_sample_plan* plans,
                                               int64_t n, const gnnshap_gcn* model, size_t* bytes) {
  Model m;
  m.gcn = model;
  if (!model) return gnnshap::fail(GNNSHAP_EINVAL, "model is NULL");
  return batch_workspace(sgs, plans, n, m, bytes);
}

extern "C" int gnnshap_explain_batch(const gnnshap_subgraph* sgs, const gnnshap_sample_plan* plans,
                                     const gnnshap_class* classes, int64_t n, const gnnshap_gcn* model,
                                     const float* X, int32_t target_class, uint64_t* masks, float* weights,
                                     float* y, float* f_empty_full, int32_t* class_out, float* phi, int32_t* info,
                                     void* ws, size_t ws_bytes, void* stream) {
  Model m;
  m.gcn = model;
  if (!model) return gnnshap::fail(GNNSHAP_EINVAL, "model is NULL");
  return explain_batch_impl(sgs, plans, classes, n, m, X, target_class, masks, weights, y, f_empty_full, class_out,
                            phi, info, ws, ws_bytes, stream);
}

extern "C" int gnnshap_gat_explain_batch_workspace(const gnnshap_subgraph* sgs, const gnnshap_sample_plan* plans,
                                                   int64_t n, const gnnshap_gat* model, size_t* bytes) {
  Model m;
  m.gat = model;
  if (!model) return gnnshap::fail(GNNSHAP_EINVAL, "model is NULL");
  return batch_workspace(sgs, plans, n, m, bytes);
}

extern "C" int gnnshap_gat_explain_batch(const gnnshap_subgraph* sgs, const gnnshap_sample_plan* plans,
                                         const gnnshap_class* classes, int64_t n, const gnnshap_gat* model,
                                         int32_t target_class, uint64_t* masks, float* weights, float* y,
                                         float* f_empty_full, int32_t* class_out, float* phi, int32_t* info,
                                         void* ws, size_t ws_bytes, void* stream) {
  Model m;
  m.gat = model;
  if (!model) return gnnshap::fail(GNNSHAP_EINVAL, "model is NULL");
  return explain_batch_impl(sgs, plans, classes, n, m, nullptr, target_class, masks, weights, y, f_empty_full,
                            class_out, phi, info, ws, ws_bytes, stream);
}
