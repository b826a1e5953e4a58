// Internal helpers shared by the library's translation units.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "gnnshap.h"

namespace gnnshap {

// Records a thread-local message and returns `status`.
int fail(int status, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();

// Bump allocator over a caller-owned workspace.  With base == nullptr it only
// measures, so the *_workspace queries and the calls share one layout.
struct Carver {
  char* base;
  size_t off = 0;
  explicit Carver(void* b) : base(static_cast<char*>(b)) {}
  template <class T>
  T* take(size_t count) {
    off = (off + 255) & ~size_t(255);
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += count * sizeof(T);
    return p;
  }
  size_t bytes() const { return (off + 255) & ~size_t(255); }
};

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Grid size for grid-stride loops: enough blocks to fill 256 CUs several times.
inline unsigned grid_for(int64_t items, int block, int64_t cap = 8192) {
  int64_t g = ceil_div(items, block);
  if (g < 1) g = 1;
  if (g > cap) g = cap;
  return static_cast<unsigned>(g);
}

// Brackets one kernel launch with two HIP events on the launch's stream when
// gnnshap_timing_begin() armed a name that prefixes `name`; inert otherwise.
class KernelTimer {
 public:
  KernelTimer(const char* name, hipStream_t s);
  ~KernelTimer();
  KernelTimer(const KernelTimer&) = delete;
  KernelTimer& operator=(const KernelTimer&) = delete;

 private:
  hipStream_t stream_;
  hipEvent_t start_ = nullptr;
  hipEvent_t stop_ = nullptr;
};

// Records an iterative solve (players, words per row, random rows,
// iterations run, sparse rows, their players) for gnnshap_timing_solves
// while timing is armed.
void timing_note_solve(int64_t M, int64_t wpr, int64_t kr, int64_t iters, int64_t rs, int64_t nnz);

// Largest dynamic LDS allocation one workgroup may request on the current device.
inline int max_lds_bytes() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 65536;
  int v = 0;
  if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess || v <= 0) v = 65536;
  return v;
}

// Page-locked staging for host-to-device copies of the calling thread: a
// ring of two buffers, each reused only after the copy that last read it has
// run (its event), so that a call never waits for earlier GPU work.
// Buffers grow on demand and are kept until the process ends.
struct HostStage {
  char* buf = nullptr;
  size_t cap = 0;
  hipEvent_t done = nullptr;
  bool pending = false;
};
// The next buffer of ring `ring` (0: batched explanation, 1: batched
// extraction), with at least `bytes`; after queueing the copy that reads it,
// record `done` on the copy's stream and set `pending`.  nullptr on failure.
HostStage* host_stage(size_t bytes, int ring);

// Copies `bytes` rounded up to a multiple of 16 (both buffers must hold the
// rounded size; both 16-byte aligned) from src to dst with a kernel on `s`,
// for copies between device memory and the page-locked buffers above: the
// copy is ordered on the stream like any kernel and never goes through the
// copy engines, whose queue can hold the host back for milliseconds when
// many copies are outstanding.  Returns a GNNSHAP status.
int copy_by_kernel(void* dst, const void* src, size_t bytes, hipStream_t s);

// Page-locked host staging of at least `bytes` for device-to-host copies of
// the calling thread (grown on demand, kept until the process ends), so the
// copy queues behind the kernels instead of blocking the host first.
// nullptr if the allocation fails.
inline void* pinned_staging(size_t bytes) {
  static thread_local void* buf = nullptr;
  static thread_local size_t cap = 0;
  if (cap < bytes) {
    if (buf) (void)hipHostFree(buf);
    buf = nullptr;
    cap = 0;
    const size_t want = bytes < 4096 ? 4096 : bytes;
    if (hipHostMalloc(&buf, want, hipHostMallocDefault) != hipSuccess) {
      (void)hipGetLastError();
      buf = nullptr;
      return nullptr;
    }
    cap = want;
  }
  return buf;
}

}  // namespace gnnshap

#define GS_HIP(call)                                                                     \
  do {                                                                                   \
    hipError_t gs_e_ = (call);                                                           \
    if (gs_e_ != hipSuccess)                                                             \
      return ::gnnshap::fail(GNNSHAP_EHIP, "%s failed: %s (%s:%d)", #call,              \
                             hipGetErrorString(gs_e_), __FILE__, __LINE__);              \
  } while (0)

#define GS_LAUNCHED() GS_HIP(hipGetLastError())

// Scope guard timing the launch(es) in the enclosing block.
#define GS_TIMED(name, stream) ::gnnshap::KernelTimer gs_kernel_timer_(name, stream)

#define GS_TRY_BEGIN try {
#define GS_TRY_END                                                               \
  }                                                                              \
  catch (...) {                                                                  \
    return ::gnnshap::fail(GNNSHAP_EHIP, "unexpected C++ exception");            \
  }
