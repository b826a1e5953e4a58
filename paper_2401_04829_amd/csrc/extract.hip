// Pruned computational graph of a target node (Sec. 3.2 and App. A of the
// GNNShap paper): BFS over in-edges to depth l, local ids by (dist, global
// id), players = in-edges of the nodes within l-1 hops, in CSR order.
//
// Device steps: one launch per BFS level (wave per frontier node, wave-
// aggregated queue appends), a two-pass compaction of the visited marks in
// global-id order (which yields the (dist, id) order without a sort), a scan
// of the destinations' in-degrees, then the player arrays.  The host waits
// once, to learn the sizes.
#include <vector>

#include "common.h"

namespace {

constexpr int kLevels = GNNSHAP_MAX_HOPS + 1;  // dist 0 .. MAX_HOPS
constexpr int kPerThread = 16;
constexpr int kChunk = 256 * kPerThread;      // marks per compaction block
constexpr int kCounters = 32;                 // int64: [0, kLevels) level sizes, [kLevels] = M

struct Ws {
  int32_t* mark;      // N: dist + 1, 0 = unvisited (zero between calls)
  int32_t* local_of;  // N: local id of a visited node
  int32_t* queue;     // N: BFS queue, level by level
  int32_t* sorted;    // N: visited nodes by (dist, id)
  int32_t* dstptr;    // N + 1
  int64_t* counters;  // kCounters
  int32_t* bcount;    // nblk * kLevels
};

Ws carve(gnnshap::Carver& c, int64_t n) {
  Ws w;
  const int64_t nblk = gnnshap::ceil_div(n, kChunk);
  w.mark = c.take<int32_t>(n);
  w.local_of = c.take<int32_t>(n);
  w.queue = c.take<int32_t>(n);
  w.sorted = c.take<int32_t>(n);
  w.dstptr = c.take<int32_t>(n + 1);
  w.counters = c.take<int64_t>(kCounters);
  w.bcount = c.take<int32_t>(nblk * kLevels);
  return w;
}

__global__ void k_init(int32_t* mark, int32_t* queue, int64_t* counters, int64_t v) {
  for (int i = 0; i < kCounters; ++i) counters[i] = 0;
  counters[0] = 1;
  mark[v] = 1;
  queue[0] = static_cast<int32_t>(v);
}

// Expands BFS level `level`: frontier = queue[begin, begin + counters[level]).
__global__ void __launch_bounds__(256) k_expand(const int64_t* __restrict__ indptr,
                                                const int32_t* __restrict__ indices,
                                                int32_t* mark, int32_t* queue,
                                                int64_t* counters, int level) {
  int64_t begin = 0;
  for (int i = 0; i < level; ++i) begin += counters[i];
  const int64_t size = counters[level];
  const int64_t end = begin + size;
  const int lane = threadIdx.x & 63;
  const int64_t wave = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = (static_cast<int64_t>(gridDim.x) * blockDim.x) >> 6;
  for (int64_t f = wave; f < size; f += nwaves) {
    const int32_t w = queue[begin + f];
    const int64_t e0 = indptr[w], e1 = indptr[w + 1];
    for (int64_t e = e0; e < e1; e += 64) {
      bool win = false;
      int32_t u = 0;
      if (e + lane < e1) {
        u = indices[e + lane];
        win = atomicCAS(&mark[u], 0, level + 2) == 0;
      }
      const uint64_t bal = __ballot(win);
      if (bal) {
        unsigned long long base = 0;
        if (lane == 0)
          base = atomicAdd(reinterpret_cast<unsigned long long*>(&counters[level + 1]),
                           static_cast<unsigned long long>(__popcll(bal)));
        base = __shfl(base, 0);
        if (win) {
          const int rank = __popcll(bal & ((1ull << lane) - 1ull));
          queue[end + static_cast<int64_t>(base) + rank] = u;
        }
      }
    }
  }
}

// Per block of kChunk marks: number of visited nodes of each level.
__global__ void __launch_bounds__(256) k_count_levels(const int32_t* __restrict__ mark, int64_t n,
                                                      int32_t* bcount, int levels) {
  __shared__ int cnt[kLevels];
  if (threadIdx.x < kLevels) cnt[threadIdx.x] = 0;
  __syncthreads();
  const int64_t base = static_cast<int64_t>(blockIdx.x) * kChunk + threadIdx.x * kPerThread;
  int m[kPerThread];
#pragma unroll
  for (int i = 0; i < kPerThread; ++i) m[i] = (base + i < n) ? mark[base + i] : 0;
  for (int l = 0; l < levels; ++l) {
    int c = 0;
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) c += (m[i] == l + 1);
    if (c) atomicAdd(&cnt[l], c);
  }
  __syncthreads();
  if (threadIdx.x < levels) bcount[static_cast<int64_t>(blockIdx.x) * kLevels + threadIdx.x] = cnt[threadIdx.x];
}

// Writes the visited nodes in (level, id) order: sorted[pos] = id, local_of[id] = pos.
__global__ void __launch_bounds__(256) k_scatter_levels(const int32_t* __restrict__ mark, int64_t n,
                                                        const int32_t* __restrict__ bcount,
                                                        const int64_t* __restrict__ counters,
                                                        int levels, int32_t* sorted,
                                                        int32_t* local_of) {
  __shared__ int64_t off[kLevels];
  __shared__ int scan[256];
  const int tid = threadIdx.x;
  if (tid < levels) {
    int64_t hb = 0;
    for (int i = 0; i < tid; ++i) hb += counters[i];
    int64_t s = 0;
    for (int64_t b = 0; b < blockIdx.x; ++b) s += bcount[b * kLevels + tid];
    off[tid] = hb + s;
  }
  const int64_t base = static_cast<int64_t>(blockIdx.x) * kChunk + tid * kPerThread;
  int m[kPerThread];
#pragma unroll
  for (int i = 0; i < kPerThread; ++i) m[i] = (base + i < n) ? mark[base + i] : 0;
  __syncthreads();
  for (int l = 0; l < levels; ++l) {
    int c = 0;
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) c += (m[i] == l + 1);
    scan[tid] = c;
    __syncthreads();
    for (int d = 1; d < 256; d <<= 1) {   // inclusive Hillis-Steele scan
      const int v = tid >= d ? scan[tid - d] : 0;
      __syncthreads();
      scan[tid] += v;
      __syncthreads();
    }
    int64_t pos = off[l] + scan[tid] - c;
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) {
      if (m[i] == l + 1) {
        const int32_t gid = static_cast<int32_t>(base + i);
        sorted[pos] = gid;
        local_of[gid] = static_cast<int32_t>(pos);
        ++pos;
      }
    }
    __syncthreads();
  }
}

// dstptr = exclusive scan of the in-degrees of the nodes within hops-1 hops;
// counters[kLevels] = M.  One block.
__global__ void __launch_bounds__(1024) k_dst_ptr(const int64_t* __restrict__ indptr,
                                                  const int32_t* __restrict__ sorted,
                                                  int64_t* counters, int hops, int32_t* dstptr) {
  __shared__ int64_t buf[1024];
  __shared__ int64_t carry;
  const int tid = threadIdx.x;
  int64_t n_dst = 0;
  for (int i = 0; i < hops; ++i) n_dst += counters[i];
  if (tid == 0) {
    carry = 0;
    dstptr[0] = 0;
  }
  __syncthreads();
  for (int64_t b0 = 0; b0 < n_dst; b0 += 1024) {
    const int64_t x = b0 + tid;
    int64_t deg = 0;
    if (x < n_dst) {
      const int32_t g = sorted[x];
      deg = indptr[g + 1] - indptr[g];
    }
    buf[tid] = deg;
    __syncthreads();
    for (int d = 1; d < 1024; d <<= 1) {
      const int64_t v = tid >= d ? buf[tid - d] : 0;
      __syncthreads();
      buf[tid] += v;
      __syncthreads();
    }
    if (x < n_dst) dstptr[x + 1] = static_cast<int32_t>(carry + buf[tid]);
    __syncthreads();
    if (tid == 1023) carry += buf[1023];
    __syncthreads();
  }
  if (tid == 0) counters[kLevels] = carry;
}

__global__ void __launch_bounds__(256) k_fill_edges(const int64_t* __restrict__ indptr,
                                                    const int32_t* __restrict__ indices,
                                                    const int32_t* __restrict__ sorted,
                                                    const int32_t* __restrict__ local_of,
                                                    const int32_t* __restrict__ dstptr,
                                                    int64_t n_dst, int32_t* edge_src,
                                                    int32_t* edge_dst, int64_t* edge_gid) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = (static_cast<int64_t>(gridDim.x) * blockDim.x) >> 6;
  for (int64_t x = wave; x < n_dst; x += nwaves) {
    const int32_t g = sorted[x];
    const int64_t e0 = indptr[g];
    const int64_t deg = indptr[g + 1] - e0;
    const int64_t out = dstptr[x];
    for (int64_t j = lane; j < deg; j += 64) {
      const int64_t e = e0 + j;
      edge_src[out + j] = local_of[indices[e]];
      edge_dst[out + j] = static_cast<int32_t>(x);
      edge_gid[out + j] = e;
    }
  }
}

// Restores the zero state of everything a call touched.
__global__ void __launch_bounds__(256) k_cleanup(Ws w, int64_t count, int64_t n_dst, int64_t nbc) {
  const int64_t t0 = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t step = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (int64_t i = t0; i < count; i += step) {
    const int32_t g = w.queue[i];
    w.mark[g] = 0;
    w.local_of[g] = 0;
    w.queue[i] = 0;
    w.sorted[i] = 0;
  }
  for (int64_t i = t0; i <= n_dst; i += step) w.dstptr[i] = 0;
  for (int64_t i = t0; i < nbc; i += step) w.bcount[i] = 0;
  for (int64_t i = t0; i < kCounters; i += step) w.counters[i] = 0;
}

// Inclusive scan of v over the 1024 threads of a block (Hillis-Steele in LDS).
__device__ __forceinline__ int64_t block_scan_1024(int64_t v, int64_t* buf) {
  const int tid = threadIdx.x;
  buf[tid] = v;
  __syncthreads();
  for (int d = 1; d < 1024; d <<= 1) {
    const int64_t t = tid >= d ? buf[tid - d] : 0;
    __syncthreads();
    buf[tid] += t;
    __syncthreads();
  }
  const int64_t r = buf[tid];
  __syncthreads();
  return r;
}

constexpr int64_t kOneBlockNodes = int64_t(1) << 18;

// The whole extraction in one workgroup (graphs of at most kOneBlockNodes
// nodes): BFS levels with a queue in the workspace, the level compaction in
// global-id order, the degree scan, the player arrays when they fit the
// caller's capacities, and the reset of the workspace.  counters[0..hops]
// receive the level sizes, counters[kLevels] = M, counters[kLevels + 1] = 1 if
// the arrays were written.
__device__ __forceinline__ void extract_one_body(const int64_t* __restrict__ indptr,
                                                 const int32_t* __restrict__ indices, int64_t n, int64_t v,
                                                 int hops, const Ws& w, int64_t cap_nodes, int64_t cap_edges,
                                                 int32_t* node_gid, int32_t* dst_ptr, int32_t* edge_src,
                                                 int32_t* edge_dst, int64_t* edge_gid, int64_t* result) {
  __shared__ int64_t lvl[kLevels + 2];     // queue offsets of the levels
  __shared__ unsigned int qcount;
  __shared__ int64_t buf[1024];
  __shared__ int64_t carry;
  __shared__ int ok;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid == 0) {
    w.mark[v] = 1;
    w.queue[0] = static_cast<int32_t>(v);
    qcount = 1;
    lvl[0] = 0;
    lvl[1] = 1;
  }
  __syncthreads();
  // BFS over in-edges, one wavefront per frontier node
  for (int level = 0; level < hops; ++level) {
    const int64_t b0 = lvl[level], b1 = lvl[level + 1];
    for (int64_t f = b0 + wave; f < b1; f += 16) {
      const int32_t node = w.queue[f];
      const int64_t e0 = indptr[node], e1 = indptr[node + 1];
      for (int64_t e = e0; e < e1; e += 64) {
        bool win = false;
        int32_t u = 0;
        if (e + lane < e1) {
          u = indices[e + lane];
          win = atomicCAS(&w.mark[u], 0, level + 2) == 0;
        }
        const uint64_t bal = __ballot(win);
        if (bal) {
          unsigned int base = 0;
          if (lane == 0) base = atomicAdd(&qcount, static_cast<unsigned int>(__popcll(bal)));
          base = __shfl(base, 0);
          if (win) w.queue[base + __popcll(bal & ((1ull << lane) - 1ull))] = u;
        }
      }
    }
    __syncthreads();
    if (tid == 0) lvl[level + 2] = qcount;
    __syncthreads();
  }
  const int64_t nodes = lvl[hops + 1];
  const int64_t n_dst = lvl[hops];
  // level compaction in global-id order: thread t scans marks [t*chunk, (t+1)*chunk)
  const int64_t chunk = (n + 1023) / 1024;
  const int64_t m0 = tid * chunk;
  const int64_t m1 = m0 + chunk < n ? m0 + chunk : n;
  for (int l = 0; l <= hops; ++l) {
    int64_t c = 0;
    for (int64_t i = m0; i < m1; ++i) c += w.mark[i] == l + 1;
    int64_t pos = lvl[l] + block_scan_1024(c, buf) - c;
    for (int64_t i = m0; i < m1 && c > 0; ++i) {
      if (w.mark[i] == l + 1) {
        w.sorted[pos] = static_cast<int32_t>(i);
        w.local_of[i] = static_cast<int32_t>(pos);
        ++pos;
        --c;
      }
    }
  }
  __syncthreads();
  // player offsets: exclusive scan of the in-degrees of the first n_dst nodes
  if (tid == 0) {
    carry = 0;
    w.dstptr[0] = 0;
  }
  __syncthreads();
  for (int64_t x0 = 0; x0 < n_dst; x0 += 1024) {
    const int64_t x = x0 + tid;
    int64_t deg = 0;
    if (x < n_dst) {
      const int32_t g = w.sorted[x];
      deg = indptr[g + 1] - indptr[g];
    }
    const int64_t incl = block_scan_1024(deg, buf);
    if (x < n_dst) w.dstptr[x + 1] = static_cast<int32_t>(carry + incl);
    __syncthreads();
    if (tid == 1023) carry += incl;
    __syncthreads();
  }
  const int64_t m = carry;
  if (tid == 0) ok = nodes <= cap_nodes && m <= cap_edges && m <= INT32_MAX;
  __syncthreads();
  if (ok) {
    for (int64_t i = tid; i < nodes; i += 1024) node_gid[i] = w.sorted[i];
    for (int64_t i = tid; i <= n_dst; i += 1024) dst_ptr[i] = w.dstptr[i];
    for (int64_t x = wave; x < n_dst; x += 16) {
      const int32_t g = w.sorted[x];
      const int64_t e0 = indptr[g];
      const int64_t deg = indptr[g + 1] - e0;
      const int64_t out = w.dstptr[x];
      for (int64_t j = lane; j < deg; j += 64) {
        const int64_t e = e0 + j;
        edge_src[out + j] = w.local_of[indices[e]];
        edge_dst[out + j] = static_cast<int32_t>(x);
        edge_gid[out + j] = e;
      }
    }
  }
  if (tid == 0) {
    for (int l = 0; l <= hops; ++l) result[l] = lvl[l + 1] - lvl[l];
    result[kLevels] = m;
    result[kLevels + 1] = ok;
  }
  __syncthreads();
  // back to the zero state (the counters are cleared after the host copy)
  for (int64_t i = tid; i < nodes; i += 1024) {
    const int32_t g = w.queue[i];
    w.mark[g] = 0;
    w.local_of[g] = 0;
    w.queue[i] = 0;
    w.sorted[i] = 0;
  }
  for (int64_t i = tid; i <= n_dst; i += 1024) w.dstptr[i] = 0;
}

__global__ void __launch_bounds__(1024) k_extract_one(const int64_t* __restrict__ indptr,
                                                      const int32_t* __restrict__ indices, int64_t n,
                                                      int64_t v, int hops, Ws w, int64_t cap_nodes,
                                                      int64_t cap_edges, int32_t* node_gid, int32_t* dst_ptr,
                                                      int32_t* edge_src, int32_t* edge_dst, int64_t* edge_gid) {
  extract_one_body(indptr, indices, n, v, hops, w, cap_nodes, cap_edges, node_gid, dst_ptr, edge_src, edge_dst,
                   edge_gid, w.counters);
}

__global__ void k_zero_counters(int64_t* counters) {
  if (threadIdx.x < kCounters) counters[threadIdx.x] = 0;
}

// ---- multi-target path --------------------------------------------------------------------

struct ExtractJob {
  int64_t v;
  int hops;
  Ws w;                    // this target's slice (zero between calls)
  int64_t cap_nodes, cap_edges;
  int32_t* node_gid;
  int32_t* dst_ptr;
  int32_t* edge_src;
  int32_t* edge_dst;
  int64_t* edge_gid;
};

// One workgroup per target; result rows of kCounters int64.
__global__ void __launch_bounds__(1024) k_extract_batch(const int64_t* __restrict__ indptr,
                                                        const int32_t* __restrict__ indices, int64_t n,
                                                        const ExtractJob* __restrict__ jobs, int64_t* results) {
  const ExtractJob J = jobs[blockIdx.x];
  extract_one_body(indptr, indices, n, J.v, J.hops, J.w, J.cap_nodes, J.cap_edges, J.node_gid, J.dst_ptr,
                   J.edge_src, J.edge_dst, J.edge_gid, results + static_cast<int64_t>(blockIdx.x) * kCounters);
}

// Batch workspace: one slice per target from the front (slice t at a fixed
// offset, zero between calls), so a workspace sized for n targets serves
// every smaller batch too.  The job table and the result rows live in
// page-locked host memory, not here.
struct BatchWs {
  char* slices;
  size_t slice_bytes;
};

size_t slice_bytes_of(int64_t num_nodes) {
  gnnshap::Carver one(nullptr);
  carve(one, num_nodes);
  return one.bytes();
}

size_t batch_bytes(int64_t num_nodes, int64_t n) { return static_cast<size_t>(n) * slice_bytes_of(num_nodes); }

BatchWs carve_batch(void* ws, int64_t num_nodes) {
  BatchWs b;
  b.slice_bytes = slice_bytes_of(num_nodes);
  b.slices = static_cast<char*>(ws);
  return b;
}

}  // namespace

extern "C" int gnnshap_extract_workspace(int64_t num_nodes, size_t* bytes) {
  gnnshap::clear_error();
  if (!bytes || num_nodes < 1) return gnnshap::fail(GNNSHAP_EINVAL, "bad arguments");
  gnnshap::Carver c(nullptr);
  carve(c, num_nodes);
  *bytes = c.bytes();
  return GNNSHAP_OK;
}

extern "C" int gnnshap_extract_subgraph(const gnnshap_graph* g, int64_t target,
                                        gnnshap_subgraph* sg, void* ws, size_t ws_bytes,
                                        void* stream) {
  GS_TRY_BEGIN
  gnnshap::clear_error();
  if (!g || !sg || !ws) return gnnshap::fail(GNNSHAP_EINVAL, "null graph, subgraph or workspace");
  if (!g->indptr || !g->indices) return gnnshap::fail(GNNSHAP_EINVAL, "null graph arrays");
  const int64_t n = g->num_nodes;
  if (n < 1 || n > INT32_MAX) return gnnshap::fail(GNNSHAP_EINVAL, "num_nodes out of range");
  if (g->num_edges < 0) return gnnshap::fail(GNNSHAP_EINVAL, "num_edges < 0");
  if (target < 0 || target >= n) return gnnshap::fail(GNNSHAP_EINVAL, "target out of range");
  const int hops = sg->num_hops;
  if (hops < 1 || hops > GNNSHAP_MAX_HOPS) return gnnshap::fail(GNNSHAP_EINVAL, "num_hops out of range");
  gnnshap::Carver need(nullptr);
  carve(need, n);
  if (ws_bytes < need.bytes())
    return gnnshap::fail(GNNSHAP_ECAPACITY, "extract workspace needs %zu bytes", need.bytes());
  gnnshap::Carver c(ws);
  const Ws w = carve(c, n);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int levels = hops + 1;
  const int64_t nblk = gnnshap::ceil_div(n, kChunk);

  if (n <= kOneBlockNodes) {
    if ((sg->cap_nodes > 0 && (!sg->node_gid || !sg->dst_ptr)) ||
        (sg->cap_edges > 0 && (!sg->edge_src || !sg->edge_dst || !sg->edge_gid)))
      return gnnshap::fail(GNNSHAP_EINVAL, "null subgraph output arrays");
    {
      GS_TIMED("k_extract_one", s);
      k_extract_one<<<1, 1024, 0, s>>>(g->indptr, g->indices, n, target, hops, w, sg->cap_nodes, sg->cap_edges,
                                       sg->node_gid, sg->dst_ptr, sg->edge_src, sg->edge_dst, sg->edge_gid);
    }
    GS_LAUNCHED();
    int64_t* h = static_cast<int64_t*>(gnnshap::pinned_staging(kCounters * sizeof(int64_t)));
    if (!h) return gnnshap::fail(GNNSHAP_EHIP, "page-locked staging allocation failed");
    GS_HIP(hipMemcpyAsync(h, w.counters, kCounters * sizeof(int64_t), hipMemcpyDeviceToHost, s));
    k_zero_counters<<<1, 64, 0, s>>>(w.counters);
    GS_LAUNCHED();
    GS_HIP(hipStreamSynchronize(s));
    int64_t nodes = 0;
    sg->hop_ptr[0] = 0;
    for (int l = 0; l < levels; ++l) {
      nodes += h[l];
      sg->hop_ptr[l + 1] = nodes;
    }
    for (int l = levels + 1; l < GNNSHAP_MAX_HOPS + 2; ++l) sg->hop_ptr[l] = nodes;
    sg->num_nodes = nodes;
    sg->num_dst = sg->hop_ptr[hops];
    sg->num_edges = h[kLevels];
    if (h[kLevels] > INT32_MAX) return gnnshap::fail(GNNSHAP_EUNSUPPORTED, "more than 2^31 players");
    if (!h[kLevels + 1])
      return gnnshap::fail(GNNSHAP_ECAPACITY, "subgraph needs %lld nodes and %lld edges", (long long)nodes,
                           (long long)h[kLevels]);
    return GNNSHAP_OK;
  }

  k_init<<<1, 1, 0, s>>>(w.mark, w.queue, w.counters, target);
  GS_LAUNCHED();
  for (int l = 0; l < hops; ++l) {
    {
      GS_TIMED("k_expand", s);
      k_expand<<<512, 256, 0, s>>>(g->indptr, g->indices, w.mark, w.queue, w.counters, l);
    }
    GS_LAUNCHED();
  }
  k_count_levels<<<static_cast<unsigned>(nblk), 256, 0, s>>>(w.mark, n, w.bcount, levels);
  GS_LAUNCHED();
  k_scatter_levels<<<static_cast<unsigned>(nblk), 256, 0, s>>>(w.mark, n, w.bcount, w.counters,
                                                                levels, w.sorted, w.local_of);
  GS_LAUNCHED();
  k_dst_ptr<<<1, 1024, 0, s>>>(g->indptr, w.sorted, w.counters, hops, w.dstptr);
  GS_LAUNCHED();

  int64_t* h = static_cast<int64_t*>(gnnshap::pinned_staging(kCounters * sizeof(int64_t)));
  if (!h) return gnnshap::fail(GNNSHAP_EHIP, "page-locked staging allocation failed");
  GS_HIP(hipMemcpyAsync(h, w.counters, kCounters * sizeof(int64_t), hipMemcpyDeviceToHost, s));
  GS_HIP(hipStreamSynchronize(s));

  int64_t nodes = 0;
  sg->hop_ptr[0] = 0;
  for (int l = 0; l < levels; ++l) {
    nodes += h[l];
    sg->hop_ptr[l + 1] = nodes;
  }
  for (int l = levels + 1; l < GNNSHAP_MAX_HOPS + 2; ++l) sg->hop_ptr[l] = nodes;
  const int64_t n_dst = sg->hop_ptr[hops];
  const int64_t m = h[kLevels];
  sg->num_nodes = nodes;
  sg->num_dst = n_dst;
  sg->num_edges = m;

  int status = GNNSHAP_OK;
  if (m > INT32_MAX) {
    status = gnnshap::fail(GNNSHAP_EUNSUPPORTED, "more than 2^31 players");
  } else if (nodes > sg->cap_nodes || m > sg->cap_edges) {
    status = gnnshap::fail(GNNSHAP_ECAPACITY, "subgraph needs %lld nodes and %lld edges",
                           (long long)nodes, (long long)m);
  } else if (!sg->node_gid || !sg->dst_ptr || (m > 0 && (!sg->edge_src || !sg->edge_dst || !sg->edge_gid))) {
    status = gnnshap::fail(GNNSHAP_EINVAL, "null subgraph output arrays");
  }
  if (status == GNNSHAP_OK) {
    GS_HIP(hipMemcpyAsync(sg->node_gid, w.sorted, nodes * sizeof(int32_t), hipMemcpyDeviceToDevice, s));
    GS_HIP(hipMemcpyAsync(sg->dst_ptr, w.dstptr, (n_dst + 1) * sizeof(int32_t), hipMemcpyDeviceToDevice, s));
    if (m > 0) {
      k_fill_edges<<<gnnshap::grid_for(n_dst * 64, 256, 4096), 256, 0, s>>>(
          g->indptr, g->indices, w.sorted, w.local_of, w.dstptr, n_dst, sg->edge_src,
          sg->edge_dst, sg->edge_gid);
      GS_LAUNCHED();
    }
  }
  k_cleanup<<<gnnshap::grid_for(std::max(nodes, nblk * kLevels), 256, 1024), 256, 0, s>>>(w, nodes, n_dst,
                                                                                         nblk * kLevels);
  GS_LAUNCHED();
  return status;
  GS_TRY_END
}

extern "C" int gnnshap_extract_batch_workspace(int64_t num_nodes, int64_t n, size_t* bytes) {
  gnnshap::clear_error();
  if (!bytes || num_nodes < 1 || n < 1) return gnnshap::fail(GNNSHAP_EINVAL, "bad arguments");
  *bytes = batch_bytes(num_nodes, n);
  return GNNSHAP_OK;
}

namespace {

// The calling thread's launched batched extraction: the kernel writes its
// result rows straight into page-locked memory (`host`), and `ready` is
// recorded behind the kernel; gnnshap_extract_batch_finish waits for it.
struct PendingExtract {
  int device = -1;
  int64_t* host = nullptr;
  size_t cap = 0;
  hipEvent_t ready = nullptr;
  int64_t n = 0;
  bool pending = false;
};

PendingExtract& pending_extract() {
  static thread_local PendingExtract p;
  return p;
}

}  // namespace

extern "C" int gnnshap_extract_batch_launch(const gnnshap_graph* g, const int64_t* targets, int64_t n,
                                            gnnshap_subgraph* sgs, void* ws, size_t ws_bytes, void* stream) {
  GS_TRY_BEGIN
  gnnshap::clear_error();
  if (!g || !targets || !sgs || !ws) return gnnshap::fail(GNNSHAP_EINVAL, "null argument");
  if (!g->indptr || !g->indices) return gnnshap::fail(GNNSHAP_EINVAL, "null graph arrays");
  const int64_t nn = g->num_nodes;
  if (nn < 1 || nn > INT32_MAX) return gnnshap::fail(GNNSHAP_EINVAL, "num_nodes out of range");
  if (n < 1 || n > INT32_MAX) return gnnshap::fail(GNNSHAP_EINVAL, "n out of range");
  if (nn > kOneBlockNodes)
    return gnnshap::fail(GNNSHAP_EUNSUPPORTED, "batched extraction supports graphs of up to %lld nodes",
                         (long long)kOneBlockNodes);
  PendingExtract& pe = pending_extract();
  if (pe.pending) return gnnshap::fail(GNNSHAP_EINVAL, "a batched extraction of this thread is not finished");
  const size_t need = batch_bytes(nn, n);
  if (ws_bytes < need) return gnnshap::fail(GNNSHAP_ECAPACITY, "batch extract workspace needs %zu bytes", need);
  const BatchWs b = carve_batch(ws, nn);
  int dev = 0;
  GS_HIP(hipGetDevice(&dev));
  if (pe.device != dev) {
    if (pe.ready) (void)hipEventDestroy(pe.ready);
    pe.ready = nullptr;
    pe.device = dev;
  }
  if (!pe.ready) GS_HIP(hipEventCreateWithFlags(&pe.ready, hipEventDisableTiming));
  const size_t hbytes = static_cast<size_t>(n) * kCounters * sizeof(int64_t);
  if (pe.cap < hbytes) {
    if (pe.host) (void)hipHostFree(pe.host);
    pe.host = nullptr;
    pe.cap = 0;
    void* hp = nullptr;
    GS_HIP(hipHostMalloc(&hp, (hbytes + 15) / 16 * 16, hipHostMallocMapped | hipHostMallocCoherent));
    pe.host = static_cast<int64_t*>(hp);
    pe.cap = hbytes;
  }
  gnnshap::HostStage* stage = gnnshap::host_stage(static_cast<size_t>(n) * sizeof(ExtractJob), 1);
  if (!stage) return gnnshap::fail(GNNSHAP_EHIP, "page-locked staging allocation failed");
  ExtractJob* jobs = reinterpret_cast<ExtractJob*>(stage->buf);
  for (int64_t t = 0; t < n; ++t) {
    const gnnshap_subgraph* sg = &sgs[t];
    if (targets[t] < 0 || targets[t] >= nn) return gnnshap::fail(GNNSHAP_EINVAL, "target %lld out of range", (long long)t);
    if (sg->num_hops < 1 || sg->num_hops > GNNSHAP_MAX_HOPS)
      return gnnshap::fail(GNNSHAP_EINVAL, "num_hops out of range in subgraph %lld", (long long)t);
    if ((sg->cap_nodes > 0 && (!sg->node_gid || !sg->dst_ptr)) ||
        (sg->cap_edges > 0 && (!sg->edge_src || !sg->edge_dst || !sg->edge_gid)))
      return gnnshap::fail(GNNSHAP_EINVAL, "null output arrays in subgraph %lld", (long long)t);
    gnnshap::Carver sc(b.slices + static_cast<size_t>(t) * b.slice_bytes);
    jobs[t] = ExtractJob{targets[t], sg->num_hops, carve(sc, nn), sg->cap_nodes, sg->cap_edges, sg->node_gid,
                         sg->dst_ptr, sg->edge_src, sg->edge_dst, sg->edge_gid};
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  // The kernel reads the job table straight from the coherent page-locked
  // staging buffer (each wavefront reads its workgroup's job once) and writes
  // the result rows straight into page-locked memory: no copy launches.
  // Every workgroup writes all the counters the host reads back; only the
  // per-target slices need to start at zero, and they reset themselves.
  {
    GS_TIMED("k_extract_batch", s);
    k_extract_batch<<<static_cast<unsigned>(n), 1024, 0, s>>>(g->indptr, g->indices, nn, jobs, pe.host);
  }
  GS_LAUNCHED();
  GS_HIP(hipEventRecord(stage->done, s));
  stage->pending = true;
  GS_HIP(hipEventRecord(pe.ready, s));
  pe.n = n;
  pe.pending = true;
  return GNNSHAP_OK;
  GS_TRY_END
}

extern "C" int gnnshap_extract_batch_finish(gnnshap_subgraph* sgs, int64_t n) {
  GS_TRY_BEGIN
  gnnshap::clear_error();
  PendingExtract& pe = pending_extract();
  if (!sgs) return gnnshap::fail(GNNSHAP_EINVAL, "null argument");
  if (!pe.pending || pe.n != n)
    return gnnshap::fail(GNNSHAP_EINVAL, "no batched extraction of %lld targets was launched by this thread",
                         (long long)n);
  // pending is cleared only once the kernel is known to be done, so that no
  // later launch frees or reuses `host` while the device may still write it
  GS_HIP(hipEventSynchronize(pe.ready));
  pe.pending = false;
  const int64_t* h = pe.host;
  bool all_ok = true;
  for (int64_t t = 0; t < n; ++t) {
    gnnshap_subgraph* sg = &sgs[t];
    const int64_t* r = h + t * kCounters;
    const int levels = sg->num_hops + 1;
    int64_t nodes = 0;
    sg->hop_ptr[0] = 0;
    for (int l = 0; l < levels; ++l) {
      nodes += r[l];
      sg->hop_ptr[l + 1] = nodes;
    }
    for (int l = levels + 1; l < GNNSHAP_MAX_HOPS + 2; ++l) sg->hop_ptr[l] = nodes;
    sg->num_nodes = nodes;
    sg->num_dst = sg->hop_ptr[sg->num_hops];
    sg->num_edges = r[kLevels];
    if (r[kLevels] > INT32_MAX) return gnnshap::fail(GNNSHAP_EUNSUPPORTED, "more than 2^31 players");
    all_ok = all_ok && r[kLevels + 1] != 0;
  }
  if (!all_ok) return gnnshap::fail(GNNSHAP_ECAPACITY, "some subgraphs exceed their capacities");
  return GNNSHAP_OK;
  GS_TRY_END
}

extern "C" int gnnshap_extract_batch(const gnnshap_graph* g, const int64_t* targets, int64_t n,
                                     gnnshap_subgraph* sgs, void* ws, size_t ws_bytes, void* stream) {
  if (int st = gnnshap_extract_batch_launch(g, targets, n, sgs, ws, ws_bytes, stream)) return st;
  return gnnshap_extract_batch_finish(sgs, n);
}

extern "C" int gnnshap_subgraph_batch_init(gnnshap_subgraph* sgs, int64_t n, int32_t num_hops, int64_t cap_nodes,
                                           int64_t cap_edges, int32_t* node_gid, int32_t* dst_ptr,
                                           int32_t* edge_src, int32_t* edge_dst, int64_t* edge_gid) {
  gnnshap::clear_error();
  if (!sgs || n < 0 || cap_nodes < 0 || cap_edges < 0) return gnnshap::fail(GNNSHAP_EINVAL, "bad argument");
  if ((cap_nodes > 0 && (!node_gid || !dst_ptr)) || (cap_edges > 0 && (!edge_src || !edge_dst || !edge_gid)))
    return gnnshap::fail(GNNSHAP_EINVAL, "null output arrays");
  for (int64_t t = 0; t < n; ++t) {
    gnnshap_subgraph& sg = sgs[t];
    sg = gnnshap_subgraph{};
    sg.num_hops = num_hops;
    sg.cap_nodes = cap_nodes;
    sg.cap_edges = cap_edges;
    sg.node_gid = node_gid ? node_gid + t * cap_nodes : nullptr;
    sg.dst_ptr = dst_ptr ? dst_ptr + t * (cap_nodes + 1) : nullptr;
    sg.edge_src = edge_src ? edge_src + t * cap_edges : nullptr;
    sg.edge_dst = edge_dst ? edge_dst + t * cap_edges : nullptr;
    sg.edge_gid = edge_gid ? edge_gid + t * cap_edges : nullptr;
  }
  return GNNSHAP_OK;
}
