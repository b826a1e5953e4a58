// Coalition sampler (Sec. 3.3.2, Alg. 3 and App. C.1 of the GNNShap paper).
//
// One wavefront per representative row.  The row is built as a bitset in
// LDS, then the row and its complement are written as packed uint64 words.
// Enumerated classes unrank their lexicographic index; random classes run
// Floyd's algorithm on Philox4x32-10 draws, 64 steps at a time: every lane
// takes one step, lanes whose draw cannot interact with an earlier step of
// the same chunk decide at once, the others are replayed in step order, so
// the result is exactly the sequential algorithm's.  Each Philox call gives
// the draws of four consecutive steps, so the words of 256 steps are made by
// one call per lane and staged in LDS.
#include <algorithm>
#include <mutex>

#include "batch.h"
#include "common.h"

namespace {

static_assert(sizeof(gnnshap_class) == 32, "class record layout");
constexpr int64_t kMaxPlayers = 131072;  // 3 bitsets of M bits in 48 KiB of LDS

struct Ws {
  gnnshap_class* classes;
};

Ws carve(gnnshap::Carver& c, int64_t ncls) {
  Ws w;
  w.classes = c.take<gnnshap_class>(ncls > 0 ? ncls : 1);
  return w;
}

// Device copy of the class table for gnnshap_sample_coalitions_noalloc: a
// fixed array in the library's code object, one per GPU, shared by every call
// on that GPU.  Host code never passes its name to a kernel or a copy (on the
// host it only stands for the symbol); it uses the device address that
// hipGetSymbolAddress returns, looked up once per device.
constexpr int64_t kScratchClasses = 16384;   // 512 KiB
__device__ __align__(256) gnnshap_class scratch[kScratchClasses];

constexpr int kMaxDevices = 64;

gnnshap_class* scratch_address() {
  static std::mutex mu;
  static gnnshap_class* addr[kMaxDevices] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    return nullptr;
  }
  std::lock_guard<std::mutex> lk(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
      (void)hipGetLastError();
      return nullptr;
    }
    addr[dev] = static_cast<gnnshap_class*>(p);
  }
  return addr[dev];
}

// Philox4x32-10 (Salmon et al., SC'11).
__device__ __forceinline__ void philox4x32_10(uint32_t& c0, uint32_t& c1, uint32_t& c2, uint32_t& c3,
                                     uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint32_t hi0 = __umulhi(0xD2511F53u, c0), lo0 = 0xD2511F53u * c0;
    const uint32_t hi1 = __umulhi(0xCD9E8D57u, c2), lo1 = 0xCD9E8D57u * c2;
    const uint32_t n0 = hi1 ^ c1 ^ k0;
    const uint32_t n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
}

// C(n, r), saturating at 2^62 (the unranked classes only need values < 2^32).
__device__ __forceinline__ uint64_t binom(int64_t n, int64_t r) {
  if (r < 0 || r > n) return 0;
  if (r > n - r) r = n - r;
  uint64_t v = 1;
  for (int64_t i = 1; i <= r; ++i) {
    const uint64_t f = static_cast<uint64_t>(n - r + i);
    if (v > (uint64_t(1) << 62) / f) return uint64_t(1) << 62;
    v = v * f / static_cast<uint64_t>(i);
  }
  return v;
}

__device__ __forceinline__ void set_bit(uint32_t* bs, int64_t j) { bs[j >> 5] |= 1u << (j & 31); }

constexpr int64_t kMaxComb = 64;   // enumerated subsets stepped incrementally up to this size

// Rows [r_begin, min(r_end, half)) of one job; one wavefront.  The class of
// the first row is found by binary search, later rows advance through the
// class table (rows are grouped by class).
__device__ __forceinline__ void sample_rows(const gnnshap::SampleJob& J, int64_t r_begin, int64_t r_end) {
  const gnnshap_class* __restrict__ cls = J.cls;
  const int64_t ncls = J.ncls, half = J.half, M = J.M, wpr = J.wpr;
  const uint32_t seed_lo = J.seed_lo, seed_hi = J.seed_hi, st_lo = J.st_lo, st_hi = J.st_hi;
  uint64_t* __restrict__ masks = J.masks;
  float* __restrict__ weights = J.weights;
  extern __shared__ uint32_t lds[];
  const int64_t nw = 2 * wpr;           // 32-bit words per bitset
  uint32_t* S = lds;                    // the row being built
  uint32_t* D1 = S + nw;                // draws seen once in the current chunk
  uint32_t* D2 = D1 + nw;               // draws seen twice or more
  const int lane = threadIdx.x;
  for (int64_t w = lane; w < nw; w += 64) {
    D1[w] = 0;
    D2[w] = 0;
  }
  if (r_end > half) r_end = half;
  int64_t lo = 0, hi = ncls - 1;        // last class starting at or before row r_begin
  while (lo < hi) {
    const int64_t mid = (lo + hi + 1) >> 1;
    if (cls[mid].row_begin <= r_begin) lo = mid; else hi = mid - 1;
  }
  gnnshap_class cur = cls[lo];
  int64_t next_begin = lo + 1 < ncls ? cls[lo + 1].row_begin : half;
  // lane 0's last enumerated subset (positions in LDS), to step to the next rank
  __shared__ int32_t comb[kMaxComb];
  __shared__ uint32_t draws[256];       // Philox words of 256 consecutive Floyd steps
  int64_t comb_cls = -1, comb_rank = -2;
  for (int64_t i = r_begin; i < r_end; ++i) {
    while (i >= next_begin) {
      ++lo;
      cur = cls[lo];
      next_begin = lo + 1 < ncls ? cls[lo + 1].row_begin : half;
    }
    const int64_t c = cur.size;
    const int full = cur.full;
    const int64_t rank = i - cur.row_begin;
    const float wt = static_cast<float>(cur.weight);
    for (int64_t w = lane; w < nw; w += 64) S[w] = 0;
    __syncthreads();
    if (full) {
      if (lane == 0) {
        if (c <= kMaxComb && comb_cls == lo && comb_rank + 1 == rank) {
          // the next c-subset in lexicographic order: bump the last position
          // that can move, restart the positions after it
          int64_t p = c - 1;
          while (comb[p] == M - c + p) --p;
          ++comb[p];
          for (int64_t q = p + 1; q < c; ++q) comb[q] = comb[q - 1] + 1;
          for (int64_t q = 0; q < c; ++q) set_bit(S, comb[q]);
        } else {
          // rank-th c-subset in lexicographic order: for each position, skip
          // whole blocks of subsets with one binary search (hockey-stick sums).
          uint64_t q = static_cast<uint64_t>(rank);
          int64_t x = 0;
          for (int64_t jj = 1; jj <= c; ++jj) {
            const int64_t r = c - jj;
            const uint64_t top = binom(M - x, r + 1);
            int64_t a = x, b = M - r - 1;
            while (a < b) {
              const int64_t mid = (a + b + 1) >> 1;
              if (top - binom(M - mid, r + 1) <= q) a = mid; else b = mid - 1;
            }
            q -= top - binom(M - a, r + 1);
            set_bit(S, a);
            if (c <= kMaxComb) comb[jj - 1] = static_cast<int32_t>(a);
            x = a + 1;
          }
        }
        comb_cls = c <= kMaxComb ? lo : -1;
        comb_rank = rank;
      }
    } else {
      for (int64_t base = 0; base < c; base += 64) {
        if ((base & 255) == 0) {
          // the draws of steps base .. base + 255: lane l evaluates counter
          // base/4 + l, whose four words are the draws of steps base + 4l + 0..3
          if (base + 4 * lane < c) {
            uint32_t c0 = static_cast<uint32_t>((base >> 2) + lane), c1 = static_cast<uint32_t>(i), c2 = st_lo,
                     c3 = st_hi;
            philox4x32_10(c0, c1, c2, c3, seed_lo, seed_hi);
            draws[4 * lane] = c0;
            draws[4 * lane + 1] = c1;
            draws[4 * lane + 2] = c2;
            draws[4 * lane + 3] = c3;
          }
          __syncthreads();
        }
        const int64_t s = base + lane;
        const bool act = s < c;
        const int64_t j = M - c + s;
        uint32_t t = 0;
        if (act) {
          const uint32_t u = draws[s & 255];
          t = static_cast<uint32_t>((static_cast<uint64_t>(u) * static_cast<uint64_t>(j + 1)) >> 32);
        }
        const int64_t wd = t >> 5;
        const uint32_t bit = 1u << (t & 31);
        if (act) {
          const uint32_t old = atomicOr(&D1[wd], bit);
          if (old & bit) atomicOr(&D2[wd], bit);
        }
        __syncthreads();
        const bool dup = act && (D2[wd] & bit);
        const bool hits_j = act && static_cast<int64_t>(t) >= M - c + base && static_cast<int64_t>(t) < j;
        const bool dirty = dup || hits_j;
        const bool in = act && !dirty && (S[wd] & bit);
        __syncthreads();
        if (act && !dirty) {
          const int64_t ins = in ? j : static_cast<int64_t>(t);
          atomicOr(&S[ins >> 5], 1u << (ins & 31));
        }
        __syncthreads();
        uint64_t todo = __ballot(dirty);
        while (todo) {                     // replay the interacting steps in order
          const int l = __ffsll(static_cast<long long>(todo)) - 1;
          todo &= todo - 1;
          const uint32_t tl = __shfl(t, l);
          if (lane == 0) {
            const int64_t jl = M - c + base + l;
            const bool inl = S[tl >> 5] & (1u << (tl & 31));
            set_bit(S, inl ? jl : static_cast<int64_t>(tl));
          }
          __syncthreads();
        }
        if (act) {
          D1[wd] = 0;
          D2[wd] = 0;
        }
        __syncthreads();
      }
    }
    __syncthreads();
    const uint64_t tail = (M & 63) ? ((uint64_t(1) << (M & 63)) - 1) : ~uint64_t(0);
    for (int64_t w = lane; w < wpr; w += 64) {
      const uint64_t word = static_cast<uint64_t>(S[2 * w]) | (static_cast<uint64_t>(S[2 * w + 1]) << 32);
      const uint64_t valid = (w == wpr - 1) ? tail : ~uint64_t(0);
      masks[i * wpr + w] = word;
      masks[(i + half) * wpr + w] = ~word & valid;
    }
    if (lane == 0) {
      weights[i] = wt;
      weights[i + half] = wt;
    }
    __syncthreads();
  }
}

// ---- one lane per row (M <= kLaneMaxPlayers) ----------------------------------------------
//
// Lane l builds row r0 + l in its own bitset (LDS word w of lane l at
// lds[64 w + l]): an enumerated row unranks its lexicographic index, a
// random row runs Floyd's algorithm step by step with the same Philox draws
// as the wavefront version, so the rows are identical.  Lanes of one class
// share the control flow.
constexpr int64_t kLaneMaxPlayers = 512;

size_t lane_lds_bytes(int64_t wpr) { return static_cast<size_t>(64 * 2 * wpr) * sizeof(uint32_t); }

__device__ __forceinline__ void sample_lane_rows(const gnnshap::SampleJob& J, int64_t r0) {
  const gnnshap_class* __restrict__ cls = J.cls;
  const int64_t ncls = J.ncls, half = J.half, M = J.M, wpr = J.wpr;
  extern __shared__ uint32_t lds[];
  const int lane = threadIdx.x;
  const int64_t i = r0 + lane;
  if (i >= half) return;
  uint32_t* B = lds + lane;              // this lane's bitset, stride 64 words
  const int64_t nw = 2 * wpr;
  for (int64_t w = 0; w < nw; ++w) B[w * 64] = 0;
  int64_t lo = 0, hi = ncls - 1;         // the class of row i
  while (lo < hi) {
    const int64_t mid = (lo + hi + 1) >> 1;
    if (cls[mid].row_begin <= i) lo = mid; else hi = mid - 1;
  }
  const gnnshap_class cur = cls[lo];
  const int64_t c = cur.size;
  const int64_t rank = i - cur.row_begin;
  if (cur.full) {
    // rank-th c-subset in lexicographic order, one position at a time
    uint64_t q = static_cast<uint64_t>(rank);
    int64_t x = 0;
    for (int64_t jj = 1; jj <= c; ++jj) {
      const int64_t r = c - jj;
      const uint64_t top = binom(M - x, r + 1);
      int64_t a = x, b = M - r - 1;
      while (a < b) {
        const int64_t mid = (a + b + 1) >> 1;
        if (top - binom(M - mid, r + 1) <= q) a = mid; else b = mid - 1;
      }
      q -= top - binom(M - a, r + 1);
      B[(a >> 5) * 64] |= 1u << (a & 31);
      x = a + 1;
    }
  } else {
    uint32_t d0 = 0, d1 = 0, d2 = 0, d3 = 0;
    for (int64_t st = 0; st < c; ++st) {
      if ((st & 3) == 0) {
        d0 = static_cast<uint32_t>(st >> 2);
        d1 = static_cast<uint32_t>(i);
        d2 = J.st_lo;
        d3 = J.st_hi;
        philox4x32_10(d0, d1, d2, d3, J.seed_lo, J.seed_hi);
      }
      const int sel = static_cast<int>(st & 3);
      const uint32_t u = sel == 0 ? d0 : sel == 1 ? d1 : sel == 2 ? d2 : d3;
      const int64_t j = M - c + st;
      const int64_t t = static_cast<int64_t>((static_cast<uint64_t>(u) * static_cast<uint64_t>(j + 1)) >> 32);
      const bool in = (B[(t >> 5) * 64] >> (t & 31)) & 1u;
      const int64_t ins = in ? j : t;
      B[(ins >> 5) * 64] |= 1u << (ins & 31);
    }
  }
  const uint64_t tail = (M & 63) ? ((uint64_t(1) << (M & 63)) - 1) : ~uint64_t(0);
  for (int64_t w = 0; w < wpr; ++w) {
    const uint64_t word = static_cast<uint64_t>(B[2 * w * 64]) | (static_cast<uint64_t>(B[(2 * w + 1) * 64]) << 32);
    const uint64_t valid = (w == wpr - 1) ? tail : ~uint64_t(0);
    J.masks[i * wpr + w] = word;
    J.masks[(i + half) * wpr + w] = ~word & valid;
  }
  const float wt = static_cast<float>(cur.weight);
  J.weights[i] = wt;
  J.weights[i + half] = wt;
}

// Consecutive representative rows per wavefront: enough workgroups to fill
// the GPU several times over, at most kRowsPerBlock rows each.
constexpr int64_t kRowsPerBlock = 16;

int64_t rows_per_block(int64_t half) {
  int64_t r = half / 4096;
  return r < 1 ? 1 : (r > kRowsPerBlock ? kRowsPerBlock : r);
}

__global__ void __launch_bounds__(64) k_sample(gnnshap::SampleJob J, int64_t rpb) {
  const int64_t r0 = static_cast<int64_t>(blockIdx.x) * rpb;
  sample_rows(J, r0, r0 + rpb);
}

__global__ void __launch_bounds__(64) k_sample_lane(gnnshap::SampleJob J) {
  sample_lane_rows(J, static_cast<int64_t>(blockIdx.x) * 64);
}

// Workgroup b takes rows [(b - blk0) rpb, + rpb) of the job with the largest
// blk0 <= b, found by a wavefront-wide search of the job table.
__global__ void __launch_bounds__(64) k_sample_batch(const gnnshap::SampleJob* __restrict__ jobs, int64_t n) {
  const int64_t b = blockIdx.x;
  const int lane = threadIdx.x;
  int64_t lo = 0, hi = n;   // jobs[lo].blk0 <= b < jobs[hi].blk0 (jobs[n].blk0 = infinity)
  while (hi - lo > 1) {
    const int64_t step = (hi - lo + 63) / 64;
    const int64_t idx = lo + lane * step;
    const bool ok = idx < hi && jobs[idx].blk0 <= b;
    const uint64_t m = __ballot(ok);
    const int64_t last = 63 - __clzll(static_cast<long long>(m));
    lo += last * step;
    hi = lo + step < hi ? lo + step : hi;
  }
  const gnnshap::SampleJob J = jobs[lo];
  const int64_t r0 = (b - J.blk0) * J.rpb;
  if (J.M <= kLaneMaxPlayers) sample_lane_rows(J, r0);
  else sample_rows(J, r0, r0 + J.rpb);
}

int check_plan(const gnnshap_sample_plan* plan) {
  if (!plan) return gnnshap::fail(GNNSHAP_EINVAL, "plan is NULL");
  if (plan->num_players < 2 || plan->num_rows < 2 || (plan->num_rows % 2) ||
      plan->words_per_row != (plan->num_players + 63) / 64 || plan->num_classes < 1)
    return gnnshap::fail(GNNSHAP_EINVAL, "plan is not the output of gnnshap_plan_samples");
  return GNNSHAP_OK;
}

}  // namespace

extern "C" int gnnshap_sample_workspace(const gnnshap_sample_plan* plan, size_t* bytes) {
  gnnshap::clear_error();
  if (!bytes) return gnnshap::fail(GNNSHAP_EINVAL, "bytes is NULL");
  if (int st = check_plan(plan)) return st;
  gnnshap::Carver c(nullptr);
  carve(c, plan->num_classes);
  *bytes = c.bytes();
  return GNNSHAP_OK;
}

namespace {

// Checks the arguments and the class table (consecutive first-half rows).
int check_sample_args(const gnnshap_sample_plan* plan, const gnnshap_class* classes, const uint64_t* masks,
                      const float* weights) {
  if (int st = check_plan(plan)) return st;
  if (!classes || !masks || !weights) return gnnshap::fail(GNNSHAP_EINVAL, "null argument");
  const int64_t M = plan->num_players;
  if (M > kMaxPlayers)
    return gnnshap::fail(GNNSHAP_EUNSUPPORTED, "sampler supports up to %lld players", (long long)kMaxPlayers);
  int64_t row = 0;
  for (int64_t i = 0; i < plan->num_classes; ++i) {
    if (classes[i].row_begin != row || classes[i].row_count < 1 || classes[i].size < 1 ||
        2 * static_cast<int64_t>(classes[i].size) > M)
      return gnnshap::fail(GNNSHAP_EINVAL, "class table inconsistent at record %lld", (long long)i);
    row += classes[i].row_count;
  }
  if (row != plan->num_rows / 2) return gnnshap::fail(GNNSHAP_EINVAL, "class table does not cover k/2 rows");
  return GNNSHAP_OK;
}

// Copies the class table to dev_classes on the stream and launches the sampler.
int sample_launch(const gnnshap_sample_plan* plan, const gnnshap_class* classes, uint64_t* masks, float* weights,
                  gnnshap_class* dev_classes, hipStream_t s) {
  const int64_t M = plan->num_players;
  const int64_t half = plan->num_rows / 2;
  Ws w;
  w.classes = dev_classes;
  GS_HIP(hipMemcpyAsync(w.classes, classes, plan->num_classes * sizeof(gnnshap_class),
                        hipMemcpyHostToDevice, s));
  const int64_t wpr = plan->words_per_row;
  if (M <= kLaneMaxPlayers) {
    const int64_t nblk = gnnshap::ceil_div(half, 64);
    if (nblk > INT32_MAX) return gnnshap::fail(GNNSHAP_EUNSUPPORTED, "too many rows");
    GS_TIMED("k_sample", s);
    const gnnshap::SampleJob job{w.classes, plan->num_classes, half, M, wpr,
                                 static_cast<uint32_t>(plan->seed), static_cast<uint32_t>(plan->seed >> 32),
                                 static_cast<uint32_t>(plan->stream_id),
                                 static_cast<uint32_t>(plan->stream_id >> 32), masks, weights, 0, 64};
    k_sample_lane<<<static_cast<unsigned>(nblk), 64, lane_lds_bytes(wpr), s>>>(job);
    GS_LAUNCHED();
    return GNNSHAP_OK;
  }
  const size_t lds = static_cast<size_t>(3 * 2 * wpr) * sizeof(uint32_t);
  const int64_t rpb = rows_per_block(half);
  const int64_t nblk = gnnshap::ceil_div(half, rpb);
  if (nblk > INT32_MAX) return gnnshap::fail(GNNSHAP_EUNSUPPORTED, "too many rows");
  const unsigned grid = static_cast<unsigned>(nblk);
  {
    GS_TIMED("k_sample", s);
    const gnnshap::SampleJob job{w.classes, plan->num_classes, half, M, wpr,
                                 static_cast<uint32_t>(plan->seed), static_cast<uint32_t>(plan->seed >> 32),
                                 static_cast<uint32_t>(plan->stream_id),
                                 static_cast<uint32_t>(plan->stream_id >> 32), masks, weights};
    k_sample<<<grid, 64, lds, s>>>(job, rpb);
  }
  GS_LAUNCHED();
  return GNNSHAP_OK;
}

}  // namespace

extern "C" int gnnshap_sample_coalitions(const gnnshap_sample_plan* plan,
                                         const gnnshap_class* classes, uint64_t* masks,
                                         float* weights, void* ws, size_t ws_bytes,
                                         void* stream) {
  GS_TRY_BEGIN
  gnnshap::clear_error();
  if (int st = check_sample_args(plan, classes, masks, weights)) return st;
  if (!ws) return gnnshap::fail(GNNSHAP_EINVAL, "null argument");
  gnnshap::Carver need(nullptr);
  carve(need, plan->num_classes);
  if (ws_bytes < need.bytes())
    return gnnshap::fail(GNNSHAP_ECAPACITY, "sample workspace needs %zu bytes", need.bytes());
  gnnshap::Carver c(ws);
  const Ws w = carve(c, plan->num_classes);
  return sample_launch(plan, classes, masks, weights, w.classes, static_cast<hipStream_t>(stream));
  GS_TRY_END
}

extern "C" int gnnshap_sample_coalitions_noalloc(const gnnshap_sample_plan* plan, const gnnshap_class* classes,
                                                 uint64_t* masks, float* weights, void* stream) {
  GS_TRY_BEGIN
  gnnshap::clear_error();
  if (int st = check_sample_args(plan, classes, masks, weights)) return st;
  if (plan->num_classes > kScratchClasses)
    return gnnshap::fail(GNNSHAP_ECAPACITY, "the allocation-free sampler holds at most %lld class records (%lld given)",
                         static_cast<long long>(kScratchClasses), static_cast<long long>(plan->num_classes));
  gnnshap_class* dev_classes = scratch_address();
  if (!dev_classes) return gnnshap::fail(GNNSHAP_EHIP, "hipGetSymbolAddress of the sampler's class table failed");
  return sample_launch(plan, classes, masks, weights, dev_classes, static_cast<hipStream_t>(stream));
  GS_TRY_END
}

int64_t gnnshap::plan_sample_batch(SampleJob* jobs, int64_t n) {
  // A row costs about (16 + M) units: the draws and bitset work of its class
  // size (up to M/2) and the words written.  Workgroups get ~1/65536 of the
  // batch's cost each, between 1 and kBatchRows rows.
  constexpr int64_t kBatchRows = 32;
  // Jobs of at most kLaneMaxPlayers players take one lane per row, 64 rows
  // per workgroup.
  double total = 0.0;
  for (int64_t t = 0; t < n; ++t)
    if (jobs[t].M > kLaneMaxPlayers) total += static_cast<double>(jobs[t].half) * (16.0 + jobs[t].M);
  const double per_block = total / 65536.0;
  int64_t blk = 0;
  for (int64_t t = 0; t < n; ++t) {
    int64_t r = static_cast<int64_t>(per_block / (16.0 + jobs[t].M));
    r = r < 1 ? 1 : (r > kBatchRows ? kBatchRows : r);
    if (jobs[t].M <= kLaneMaxPlayers) r = 64;
    jobs[t].rpb = r;
    jobs[t].blk0 = blk;
    blk += ceil_div(jobs[t].half, r);
  }
  return blk;
}

int gnnshap::launch_sample_batch(const SampleJob* jobs, int64_t n, int64_t blocks, int64_t max_wpr, hipStream_t s) {
  if (n < 1) return GNNSHAP_OK;
  if (blocks > INT32_MAX) return fail(GNNSHAP_EUNSUPPORTED, "too many rows");
  const size_t lds = std::max(static_cast<size_t>(3 * 2 * max_wpr) * sizeof(uint32_t),
                              lane_lds_bytes(std::min<int64_t>(max_wpr, kLaneMaxPlayers / 64)));
  GS_TIMED("k_sample_batch", s);
  k_sample_batch<<<static_cast<unsigned>(blocks), 64, lds, s>>>(jobs, n);
  GS_LAUNCHED();
  return GNNSHAP_OK;
}
