// HIP-event timing of one named kernel (diagnostics for measurements).
#include <algorithm>
#include <atomic>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "common.h"

namespace gnnshap {
namespace {
std::atomic<bool> g_on{false};
std::mutex g_mu;
std::string g_name;
std::vector<std::pair<hipEvent_t, hipEvent_t>> g_recs;
std::vector<int64_t> g_solves;   // 6 per iterative solve while armed
}  // namespace

void timing_note_solve(int64_t M, int64_t wpr, int64_t kr, int64_t iters, int64_t rs, int64_t nnz) {
  if (!g_on.load(std::memory_order_relaxed)) return;
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_on.load()) return;
  g_solves.insert(g_solves.end(), {M, wpr, kr, iters, rs, nnz});
}

KernelTimer::KernelTimer(const char* name, hipStream_t s) : stream_(s) {
  if (!g_on.load(std::memory_order_relaxed)) return;
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_on.load() || std::strncmp(name, g_name.c_str(), g_name.size()) != 0) return;
  if (hipEventCreate(&start_) != hipSuccess || hipEventCreate(&stop_) != hipSuccess ||
      hipEventRecord(start_, s) != hipSuccess) {
    start_ = stop_ = nullptr;
    (void)hipGetLastError();
  }
}

KernelTimer::~KernelTimer() {
  if (!start_) return;
  if (hipEventRecord(stop_, stream_) != hipSuccess) {
    (void)hipGetLastError();
    return;
  }
  std::lock_guard<std::mutex> lk(g_mu);
  g_recs.emplace_back(start_, stop_);
}

}  // namespace gnnshap

extern "C" int gnnshap_timing_begin(const char* kernel_name) {
  gnnshap::clear_error();
  if (!kernel_name || !kernel_name[0]) return gnnshap::fail(GNNSHAP_EINVAL, "empty kernel name");
  std::lock_guard<std::mutex> lk(gnnshap::g_mu);
  if (gnnshap::g_on.load()) return gnnshap::fail(GNNSHAP_EINVAL, "timing already armed");
  gnnshap::g_name = kernel_name;
  gnnshap::g_recs.clear();
  gnnshap::g_solves.clear();
  gnnshap::g_on.store(true);
  return GNNSHAP_OK;
}

extern "C" int gnnshap_timing_end(double* total_ms, int64_t* launches) {
  gnnshap::clear_error();
  std::vector<std::pair<hipEvent_t, hipEvent_t>> recs;
  {
    std::lock_guard<std::mutex> lk(gnnshap::g_mu);
    gnnshap::g_on.store(false);
    recs.swap(gnnshap::g_recs);
  }
  double total = 0.0;
  int status = GNNSHAP_OK;
  for (auto& r : recs) {
    float ms = 0.f;
    if (hipEventSynchronize(r.second) == hipSuccess && hipEventElapsedTime(&ms, r.first, r.second) == hipSuccess)
      total += ms;
    else
      status = gnnshap::fail(GNNSHAP_EHIP, "event timing failed: %s", hipGetErrorString(hipGetLastError()));
    (void)hipEventDestroy(r.first);
    (void)hipEventDestroy(r.second);
  }
  if (total_ms) *total_ms = total;
  if (launches) *launches = static_cast<int64_t>(recs.size());
  return status;
}

extern "C" int gnnshap_timing_solves(int64_t* records, int64_t cap, int64_t* count) {
  gnnshap::clear_error();
  if (!count || cap < 0 || (cap > 0 && !records)) return gnnshap::fail(GNNSHAP_EINVAL, "bad arguments");
  std::lock_guard<std::mutex> lk(gnnshap::g_mu);
  const int64_t n = static_cast<int64_t>(gnnshap::g_solves.size() / 6);
  *count = n;
  if (cap < n) return gnnshap::fail(GNNSHAP_ECAPACITY, "%lld solve records", static_cast<long long>(n));
  std::copy(gnnshap::g_solves.begin(), gnnshap::g_solves.end(), records);
  return GNNSHAP_OK;
}
