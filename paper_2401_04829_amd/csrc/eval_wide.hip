// Coalition values of a two-layer GCN with a wide hidden layer, on bf16 MFMA
// over an exact split of the fp32 operand (Sec. 3.4 of the GNNShap paper;
// the GCN of Sec. 4.2).
//
// With two hops, H_1 = {v} and v's in-neighbours are the only nodes that
// players enter.  Under coalition c, layer 1 at x in H_1 is
//   H^1_c[x] = relu( d_c(x)^-1/2 ( sum_{e -> x, e in c} d_c(src e)^-1/2 Z[src e] + d_c(x)^-1/2 Z[x] ) + b_1 ),
// Z = X W_1, d = 1 + in-degree under c; y_c = H^2_c[v, class] is
//   d_c(v)^-1/2 ( sum_{e -> v, e in c} d_c(src e)^-1/2 t_c[src e] + d_c(v)^-1/2 t_c[v] ) + b_2,
// t_c[x] = H^1_c[x] . W_2[:, class].
// A source outside H_1 has no players entering it, so its degree is 1 under
// every coalition: for those players the sum is a 0/1 contraction
//   D_c[f] = sum_e [e in c] Z[src e][f],
// a (features x players) x (players x coalitions) product with the mask bits
// as the right operand.  The mask bits are exact in bf16 and each fp32 value
// of Z is the exact sum of three bf16 parts (hi + mid + lo, 8 significant
// bits each), so the product runs on v_mfma_f32_16x16x32_bf16, three per
// operand tile, with fp32 accumulation: the same sums as an fp32 product at
// a sixteenth of the MFMA cycles per flop.  The few players
// whose source lies in H_1 (the in-edges of v, the edge v -> x, edges between
// in-neighbours) carry a coalition-dependent d^-1/2 and are added in the
// epilogue.  For the sampler's complement pairs (row b + k/2 = NOT row b),
// D of the complement is S - D_c with S the sum over all those players, so
// only the first half of the rows is contracted.
//
// Kernels, per target:
//   k_wide_ends_l1, k_wide_ends_out
//                the two end coalitions (no players, every player) for every
//                class, and the explained class: layer 1 at every node of H_1
//                as partial sums by four workgroups per (node, 64 features),
//                then in one workgroup the sums, layer 1's end and layer 2 by
//                one wavefront per class
//   k_wide_prep  one workgroup: operand-unit offsets of each node and the
//                list of players whose source is in H_1
//   k_wide_zop   the A operands: for 32 players (one unit) and 16 features
//                (one tile), lane (r, g) of a wavefront holds Z[src][f] for
//                feature 16 tile + r and players 8 g .. 8 g + 7, as three
//                uint4 of eight bf16 (hi, mid, lo; zero for padding and for
//                the players above)
//   k_wide_sum   S (pairs only): per node and feature, fixed summation order
//   k_wide_deg   in-degree of every node of H_1 under every contracted row
//   k_wide_l1    one workgroup per (node, 256 coalitions, 64 features):
//                four wavefronts of 64 coalitions, 4 x 4 16x16 output tiles
//                each; then the epilogue to t_c[x] (and the complement's)
//   k_wide_out   y per row from t, the degrees and the mask bits of v's in-edges
#include "wide.h"

namespace {

typedef float mx4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf8_t __attribute__((ext_vector_type(8)));

constexpr int kWaves = 4;                      // wavefronts per workgroup
constexpr int kWaveRows = 64;                  // coalitions per wavefront (four tiles of 16)
constexpr int kBlockRows = kWaves * kWaveRows;
constexpr int kTiles = 4;                      // 16-feature tiles per workgroup
constexpr int kUnit = 32;                      // players per operand unit (one bf16 MFMA step)
constexpr int kParts = 3;                      // bf16 parts of an fp32 operand: hi + mid + lo

// fp32 -> bf16 bits, rounded to nearest even (finite inputs).
__device__ __forceinline__ uint32_t bf16_bits(float x) {
  const uint32_t u = __float_as_uint(x);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ float bf16_value(uint32_t b) { return __uint_as_float(b << 16); }

__global__ void __launch_bounds__(1024) k_wide_prep(const int32_t* __restrict__ dst_ptr,
                                                    const int32_t* __restrict__ edge_src, int64_t n1,
                                                    int32_t* __restrict__ seg, int32_t* __restrict__ spec_ptr,
                                                    int32_t* __restrict__ spec_e) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nwaves = blockDim.x >> 6;
  // counts: one wavefront per node
  for (int64_t x = wave; x < n1; x += nwaves) {
    const int e0 = dst_ptr[x], e1 = dst_ptr[x + 1];
    int cnt = 0;
    for (int b = e0; b < e1; b += 64) {
      const int e = b + lane;
      const bool sp = e < e1 && edge_src[e] < n1;
      cnt += __popcll(__ballot(sp));
    }
    if (lane == 0) {
      spec_ptr[x + 1] = cnt;
      seg[x + 1] = (e1 - e0 + kUnit - 1) / kUnit;
    }
  }
  __syncthreads();
  if (tid == 0) {
    seg[0] = 0;
    spec_ptr[0] = 0;
    for (int64_t x = 0; x < n1; ++x) {
      seg[x + 1] += seg[x];
      spec_ptr[x + 1] += spec_ptr[x];
    }
  }
  __syncthreads();
  // lists in player order
  for (int64_t x = wave; x < n1; x += nwaves) {
    const int e0 = dst_ptr[x], e1 = dst_ptr[x + 1];
    int out = spec_ptr[x];
    for (int b = e0; b < e1; b += 64) {
      const int e = b + lane;
      const bool sp = e < e1 && edge_src[e] < n1;
      const uint64_t m = __ballot(sp);
      if (sp) spec_e[out + __popcll(m & ((uint64_t(1) << lane) - 1))] = e;
      out += __popcll(m);
    }
  }
}

// The A operands in bf16 parts: for unit U (32 players of one node), feature
// tile ft and lane (r, g), the eight values Z[src][16 ft + r] of players
// 8 g .. 8 g + 7 of the unit (zero for padding and for sources in H_1),
// each split into hi + mid + lo (round to nearest at each step, so the three
// parts add up to the fp32 value exactly), stored as three uint4 of eight
// bf16: part p of (U, ft) at Zop[((U ntot + ft) kParts + p) 64 + lane].
// The units of nodes 0 .. nn - 1 (a prefix of H_1) are built.
__global__ void __launch_bounds__(256) k_wide_zop(const int32_t* __restrict__ dst_ptr,
                                                  const int32_t* __restrict__ edge_src, int64_t n1, int64_t nn,
                                                  const int32_t* __restrict__ seg, const float* __restrict__ Zc, int h,
                                                  int ntot, int64_t units_cap, uint4* __restrict__ Zop) {
  const int64_t units = seg[nn];
  const int64_t total = units * ntot * 64;
  for (int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; idx < total;
       idx += static_cast<int64_t>(gridDim.x) * 256) {
    const int lane = static_cast<int>(idx & 63);
    const int64_t rest = idx >> 6;
    const int ft = static_cast<int>(rest % ntot);
    const int64_t U = rest / ntot;
    if (U >= units_cap) break;
    int64_t lo = 0, hi = nn;                    // node x with seg[x] <= U < seg[x + 1]
    while (hi - lo > 1) {
      const int64_t mid = (lo + hi) >> 1;
      if (seg[mid] <= U) lo = mid;
      else hi = mid;
    }
    const int64_t x = lo;
    const int e0 = dst_ptr[x], e1 = dst_ptr[x + 1];
    const int base = e0 + static_cast<int>(U - seg[x]) * kUnit;
    const int f = 16 * ft + (lane & 15), g = lane >> 4;
    uint32_t w[kParts][4];
#pragma unroll
    for (int t = 0; t < 8; t += 2) {
      uint32_t pb[kParts][2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int e = base + 8 * g + t + i;
        const int32_t u = e < e1 ? edge_src[e] : 0;
        const float v = (e < e1 && u >= n1) ? Zc[static_cast<int64_t>(u) * h + f] : 0.f;
        const uint32_t b0 = bf16_bits(v);
        const float r1 = v - bf16_value(b0);
        const uint32_t b1 = bf16_bits(r1);
        const uint32_t b2 = bf16_bits(r1 - bf16_value(b1));
        pb[0][i] = b0;
        pb[1][i] = b1;
        pb[2][i] = b2;
      }
#pragma unroll
      for (int p = 0; p < kParts; ++p) w[p][t / 2] = pb[p][0] | (pb[p][1] << 16);
    }
#pragma unroll
    for (int p = 0; p < kParts; ++p)
      Zop[(rest * kParts + p) * 64 + lane] = make_uint4(w[p][0], w[p][1], w[p][2], w[p][3]);
  }
}

// S[x][f] = sum of Z[src e][f] over the players e -> x whose source is not in
// H_1: thread (j, r) of the workgroup (1024 threads) sums the players j,
// j + 64, ... for feature 16 tile + r (four loads in flight), then the 64
// partial sums are added in a fixed tree.
__global__ void __launch_bounds__(1024) k_wide_sum(const int32_t* __restrict__ dst_ptr,
                                                   const int32_t* __restrict__ edge_src, int64_t n1,
                                                   const float* __restrict__ Zc, int h, int ntot,
                                                   float* __restrict__ S) {
  __shared__ float part[64][17];
  const int64_t x = blockIdx.x / ntot;
  const int ft = static_cast<int>(blockIdx.x % ntot);
  const int r = threadIdx.x & 15, j = threadIdx.x >> 4;
  const int f = 16 * ft + r;
  const int e0 = dst_ptr[x], e1 = dst_ptr[x + 1];
  float a4[4] = {0.f, 0.f, 0.f, 0.f};
  for (int e = e0 + j; e < e1; e += 256) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int eq = e + 64 * q;
      const int32_t u = eq < e1 ? edge_src[eq] : 0;
      if (eq < e1 && u >= n1) a4[q] += Zc[static_cast<int64_t>(u) * h + f];
    }
  }
  part[j][r] = (a4[0] + a4[1]) + (a4[2] + a4[3]);
  __syncthreads();
  for (int w = 32; w >= 1; w >>= 1) {
    if (j < w) part[j][r] += part[j + w][r];
    __syncthreads();
  }
  if (j == 0) S[x * h + f] = part[0][r];
}

// deg[b][x] = number of row b's players entering x, b < nrows, x < n1.
__global__ void __launch_bounds__(256) k_wide_deg(const uint64_t* __restrict__ masks, int64_t wpr, int64_t nrows,
                                                  const int32_t* __restrict__ dst_ptr, int64_t n1,
                                                  int32_t* __restrict__ deg) {
  const int64_t total = nrows * n1;
  for (int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; idx < total;
       idx += static_cast<int64_t>(gridDim.x) * 256) {
    const int64_t b = idx / n1, x = idx % n1;
    const uint64_t* mr = masks + b * wpr;
    const int64_t e0 = dst_ptr[x], e1 = dst_ptr[x + 1];
    int cnt = 0;
    for (int64_t w = e0 >> 6; e1 > e0 && w <= ((e1 - 1) >> 6); ++w) {
      uint64_t word = mr[w];
      const int64_t lo = w * 64;
      if (e0 > lo) word &= ~uint64_t(0) << (e0 - lo);
      if (e1 < lo + 64) word &= (uint64_t(1) << (e1 - lo)) - 1;
      cnt += __popcll(word);
    }
    deg[idx] = cnt;
  }
}

// What the epilogue of the contraction makes of a layer's sums at x:
//   kProj   H at x projected on the explained class's column of the next
//           weight matrix (the last hidden layer): t[fb][row][x]
//   kFull   H at x itself (layer 1 of a three-layer model): Hout rows
// and where the players whose source is in H_1 (and x's self loop) take
// their input row from: Zc (constant, layer 1) or Zrow (the coalition's
// own rows, layer 2 of a three-layer model: kProjRows).
enum : int { kProj = 0, kFull = 1, kProjRows = 2 };

// One layer at node x = blockIdx.x / cblocks of H_1 for 256 coalitions
// (block blockIdx.x % cblocks of the pass's nloc rows r0 .. r0 + nloc - 1)
// and features 64 blockIdx.y .. + 63.  Wavefront w holds pass rows c0 ..
// c0 + 63, c0 = 256 block + 64 w, as four 16-row tiles; lane (r, g) = (lane
// % 16, lane / 16) holds, per tile ct and feature tile ft, features 16 ft +
// 4 g .. + 3 of pass row c0 + 16 ct + r.  The row's complement (pairs) is
// row + khalf; per-row arrays of the pass (Hout, Zrow: [pass row][x][f])
// hold the complement of pass row i at i + nloc.
template <bool PAIRS, int MODE>
__global__ void __launch_bounds__(kBlockRows, 2) k_wide_l1(
    const uint64_t* __restrict__ masks, int64_t wpr, int64_t r0, int64_t nloc, int64_t khalf, int64_t cblocks,
    const int32_t* __restrict__ dst_ptr, const int32_t* __restrict__ edge_src, int64_t n1,
    const int32_t* __restrict__ seg, const uint4* __restrict__ Zop, int ntot, int h, const float* __restrict__ Zc,
    const float* __restrict__ S, const int32_t* __restrict__ spec_ptr, const int32_t* __restrict__ spec_e,
    const int32_t* __restrict__ deg, const float* __restrict__ b1, const float* __restrict__ W2, int C,
    const int32_t* __restrict__ ctl, float* __restrict__ t, int64_t k, const float* __restrict__ Zrow,
    float* __restrict__ Hout) {
  const int64_t x = blockIdx.x / cblocks;
  const int64_t cb = blockIdx.x % cblocks;
  const int fb = blockIdx.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, rl = lane & 15, g = lane >> 4;
  const int64_t c0 = cb * kBlockRows + wave * kWaveRows;
  if (c0 >= nloc) return;                        // no barrier in this kernel
  const int e0 = dst_ptr[x], e1 = dst_ptr[x + 1];
  const int u0 = seg[x], nu = seg[x + 1] - u0;
  const int ft0 = fb * kTiles;
  const int nt = ntot - ft0 < kTiles ? ntot - ft0 : kTiles;

  int64_t row[4], lr[4];   // the mask row and the pass row of each tile (clamped to 0 when invalid)
  bool valid[4];
#pragma unroll
  for (int ct = 0; ct < 4; ++ct) {
    const int64_t i = c0 + 16 * ct + rl;
    valid[ct] = i < nloc;
    lr[ct] = valid[ct] ? i : 0;
    row[ct] = r0 + lr[ct];
  }
  mx4_t D[4][kTiles];
#pragma unroll
  for (int ct = 0; ct < 4; ++ct)
#pragma unroll
    for (int ft = 0; ft < kTiles; ++ft) D[ct][ft] = mx4_t{0.f, 0.f, 0.f, 0.f};

  // A operands of unit q: lane's three parts for each of the kTiles feature
  // tiles; the next unit's are loaded while this one is multiplied
  const int64_t ustride = static_cast<int64_t>(ntot) * kParts * 64;
  const uint4* zp = Zop + static_cast<int64_t>(u0) * ustride + static_cast<int64_t>(ft0) * kParts * 64 + lane;
  // (every load is of a valid unit and tile: the last unit's successor and
  // the tiles beyond nt repeat a valid one, whose products are not used)
  uint4 a[kTiles][kParts], an[kTiles][kParts];
  if (nu > 0) {
#pragma unroll
    for (int ft = 0; ft < kTiles; ++ft)
#pragma unroll
      for (int p = 0; p < kParts; ++p) a[ft][p] = zp[((ft < nt ? ft : nt - 1) * kParts + p) * 64];
  }
  // the mask bits of 64 players (units q, q + 1) of each of the lane's rows;
  // the window of the next two units is loaded while these are multiplied
  auto window = [&](int q, int ct) -> uint64_t {
    if (!valid[ct] || q >= nu) return 0;
    const int64_t pb = e0 + static_cast<int64_t>(kUnit) * q;
    const int64_t wa = pb >> 6;
    const int sh = static_cast<int>(pb & 63);
    const uint64_t* mr = masks + row[ct] * wpr;
    const uint64_t lo = mr[wa];
    const uint64_t hi = (sh && wa + 1 < wpr) ? mr[wa + 1] : 0;
    return sh ? (lo >> sh) | (hi << (64 - sh)) : lo;
  };
  uint64_t win[4], wnext[4];
#pragma unroll
  for (int ct = 0; ct < 4; ++ct) wnext[ct] = window(0, ct);
  for (int q = 0; q < nu; ++q) {
    if ((q & 1) == 0) {
#pragma unroll
      for (int ct = 0; ct < 4; ++ct) {
        win[ct] = wnext[ct];
        wnext[ct] = window(q + 2, ct);
      }
    }
    const int64_t qn = q + 1 < nu ? q + 1 : q;
#pragma unroll
    for (int ft = 0; ft < kTiles; ++ft)
#pragma unroll
      for (int p = 0; p < kParts; ++p) an[ft][p] = zp[qn * ustride + ((ft < nt ? ft : nt - 1) * kParts + p) * 64];
    // B: the lane's eight players 8 g .. 8 g + 7 of the unit for row 16 ct +
    // rl, as eight bf16 of 0.0 or 1.0 (0x3F80), two per dword
#pragma unroll
    for (int ct = 0; ct < 4; ++ct) {
      const uint32_t byte = static_cast<uint32_t>(win[ct] >> (32 * (q & 1) + 8 * g)) & 0xffu;
      uint32_t bw[4];
#pragma unroll
      for (int t = 0; t < 4; ++t)
        bw[t] = (((byte >> (2 * t)) & 1u) | (((byte >> (2 * t + 1)) & 1u) << 16)) * 0x3F80u;
      const bf8_t bv = __builtin_bit_cast(bf8_t, make_uint4(bw[0], bw[1], bw[2], bw[3]));
      // (tiles beyond nt multiply a repeated valid tile; the epilogue skips them)
#pragma unroll
      for (int ft = 0; ft < kTiles; ++ft)
#pragma unroll
        for (int p = 0; p < kParts; ++p)
          D[ct][ft] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf8_t, a[ft][p]), bv, D[ct][ft],
                                                              0, 0, 0);
    }
#pragma unroll
    for (int ft = 0; ft < kTiles; ++ft)
#pragma unroll
      for (int p = 0; p < kParts; ++p) a[ft][p] = an[ft][p];
  }

  // epilogue: the players whose source is in H_1, self loop, bias, ReLU and
  // (kProj, kProjRows) the explained class's column of the next weight
  // matrix, per row (and its complement).  The player loop runs once for the
  // four row tiles: its source, the source's size and (constant input rows)
  // its feature values are loaded once, each row tile adds them with its own
  // coefficient (0 for the coalition it is not in).
  const int cls = MODE == kFull ? 0 : ctl[0];
  const int nx = e1 - e0;
  const int sp0 = spec_ptr[x], sp1 = spec_ptr[x + 1];
  const int32_t* dgr[4];
  const uint64_t* mrr[4];
#pragma unroll
  for (int ct = 0; ct < 4; ++ct) {
    const int64_t rr = valid[ct] ? row[ct] : 0;
    dgr[ct] = deg + rr * n1;
    mrr[ct] = masks + rr * wpr;
  }
  mx4_t P[4][kTiles];   // the complement's sums (pairs)
#pragma unroll
  for (int ft = 0; ft < kTiles; ++ft) {
    const int f = 16 * (ft0 + (ft < nt ? ft : nt - 1)) + 4 * g;
    const float4 s4 = PAIRS ? *reinterpret_cast<const float4*>(S + x * h + f) : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int ct = 0; ct < 4; ++ct)
      P[ct][ft] = mx4_t{s4.x - D[ct][ft][0], s4.y - D[ct][ft][1], s4.z - D[ct][ft][2], s4.w - D[ct][ft][3]};
  }
  for (int sp = sp0; sp < sp1; ++sp) {
    const int e = spec_e[sp];
    const int32_t u = edge_src[e];
    const int nuu = PAIRS ? dst_ptr[u + 1] - dst_ptr[u] : 0;
    float cw[4], cp[4];
#pragma unroll
    for (int ct = 0; ct < 4; ++ct) {
      const bool bit = (mrr[ct][e >> 6] >> (e & 63)) & 1;
      const int du = dgr[ct][u];
      cw[ct] = bit ? __builtin_amdgcn_rsqf(1.0f + static_cast<float>(du)) : 0.f;
      cp[ct] = (PAIRS && !bit) ? __builtin_amdgcn_rsqf(1.0f + static_cast<float>(nuu - du)) : 0.f;
    }
#pragma unroll
    for (int ft = 0; ft < kTiles; ++ft) {
      if (ft >= nt) continue;
      const int f = 16 * (ft0 + ft) + 4 * g;
      if (MODE != kProjRows) {
        const float4 zu = *reinterpret_cast<const float4*>(Zc + static_cast<int64_t>(u) * h + f);
#pragma unroll
        for (int ct = 0; ct < 4; ++ct) {
          D[ct][ft][0] = fmaf(cw[ct], zu.x, D[ct][ft][0]);
          D[ct][ft][1] = fmaf(cw[ct], zu.y, D[ct][ft][1]);
          D[ct][ft][2] = fmaf(cw[ct], zu.z, D[ct][ft][2]);
          D[ct][ft][3] = fmaf(cw[ct], zu.w, D[ct][ft][3]);
          if (PAIRS) {
            P[ct][ft][0] = fmaf(cp[ct], zu.x, P[ct][ft][0]);
            P[ct][ft][1] = fmaf(cp[ct], zu.y, P[ct][ft][1]);
            P[ct][ft][2] = fmaf(cp[ct], zu.z, P[ct][ft][2]);
            P[ct][ft][3] = fmaf(cp[ct], zu.w, P[ct][ft][3]);
          }
        }
      } else {
        // the source's row under the coalition that holds the player (the
        // row itself, or with pairs its complement): one load, no branch, so
        // the loads of the four row tiles go out together; the other
        // coefficient is 0 and adds nothing
#pragma unroll
        for (int ct = 0; ct < 4; ++ct) {
          const bool own = !PAIRS || cw[ct] != 0.f;
          const float4 zu =
              *reinterpret_cast<const float4*>(Zrow + ((own ? lr[ct] : lr[ct] + nloc) * n1 + u) * h + f);
          D[ct][ft][0] = fmaf(cw[ct], zu.x, D[ct][ft][0]);
          D[ct][ft][1] = fmaf(cw[ct], zu.y, D[ct][ft][1]);
          D[ct][ft][2] = fmaf(cw[ct], zu.z, D[ct][ft][2]);
          D[ct][ft][3] = fmaf(cw[ct], zu.w, D[ct][ft][3]);
          if (PAIRS) {
            P[ct][ft][0] = fmaf(cp[ct], zu.x, P[ct][ft][0]);
            P[ct][ft][1] = fmaf(cp[ct], zu.y, P[ct][ft][1]);
            P[ct][ft][2] = fmaf(cp[ct], zu.z, P[ct][ft][2]);
            P[ct][ft][3] = fmaf(cp[ct], zu.w, P[ct][ft][3]);
          }
        }
      }
    }
  }
#pragma unroll
  for (int ct = 0; ct < 4; ++ct) {
    const int dgx = dgr[ct][x];
    const float dx = __builtin_amdgcn_rsqf(1.0f + static_cast<float>(dgx));
    const float dxp = __builtin_amdgcn_rsqf(1.0f + static_cast<float>(nx - dgx));
    if (MODE == kFull) {
      // H at x, and at x under the complement, as rows of the pass
#pragma unroll
      for (int ft = 0; ft < kTiles; ++ft) {
        if (ft >= nt) continue;
        const int f = 16 * (ft0 + ft) + 4 * g;
        const float4 zx = *reinterpret_cast<const float4*>(Zc + x * h + f);
        const float zxv[4] = {zx.x, zx.y, zx.z, zx.w};
        float hv[4], hp[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float bb = b1 ? b1[f + i] : 0.f;
          hv[i] = fmaxf(fmaf(dx, fmaf(dx, zxv[i], D[ct][ft][i]), bb), 0.f);
          hp[i] = PAIRS ? fmaxf(fmaf(dxp, fmaf(dxp, zxv[i], P[ct][ft][i]), bb), 0.f) : 0.f;
        }
        if (valid[ct]) {
          *reinterpret_cast<float4*>(Hout + (lr[ct] * n1 + x) * h + f) = make_float4(hv[0], hv[1], hv[2], hv[3]);
          if (PAIRS)
            *reinterpret_cast<float4*>(Hout + ((lr[ct] + nloc) * n1 + x) * h + f) =
                make_float4(hp[0], hp[1], hp[2], hp[3]);
        }
      }
      continue;
    }
    float tc = 0.f, tcp = 0.f;
#pragma unroll
    for (int ft = 0; ft < kTiles; ++ft) {
      if (ft >= nt) continue;
      const int f = 16 * (ft0 + ft) + 4 * g;
      // the self loop's input row: constant, or the coalition's own (and its complement's)
      const float4 zx = MODE == kProjRows ? *reinterpret_cast<const float4*>(Zrow + (lr[ct] * n1 + x) * h + f)
                                          : *reinterpret_cast<const float4*>(Zc + x * h + f);
      const float4 zxc = (MODE == kProjRows && PAIRS)
                             ? *reinterpret_cast<const float4*>(Zrow + ((lr[ct] + nloc) * n1 + x) * h + f)
                             : zx;
      const float zxv[4] = {zx.x, zx.y, zx.z, zx.w};
      const float zxcv[4] = {zxc.x, zxc.y, zxc.z, zxc.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float bb = b1 ? b1[f + i] : 0.f;
        const float ww = W2[static_cast<int64_t>(f + i) * C + cls];
        tc = fmaf(fmaxf(fmaf(dx, fmaf(dx, zxv[i], D[ct][ft][i]), bb), 0.f), ww, tc);
        if (PAIRS) tcp = fmaf(fmaxf(fmaf(dxp, fmaf(dxp, zxcv[i], P[ct][ft][i]), bb), 0.f), ww, tcp);
      }
    }
    tc += __shfl_xor(tc, 16);
    tc += __shfl_xor(tc, 32);
    if (PAIRS) {
      tcp += __shfl_xor(tcp, 16);
      tcp += __shfl_xor(tcp, 32);
    }
    if (valid[ct] && g == 0) {
      t[(static_cast<int64_t>(fb) * k + row[ct]) * n1 + x] = tc;
      if (PAIRS) t[(static_cast<int64_t>(fb) * k + row[ct] + khalf) * n1 + x] = tcp;
    }
  }
}

// y of row b (b < nrows) and, with pairs, of its complement b + khalf.
// Node x of 1 .. n_in - 1 (the first hop) is the source of the target's
// player x - 1 (the extraction orders both by global id).
template <bool PAIRS>
__global__ void __launch_bounds__(256) k_wide_out(const uint64_t* __restrict__ masks, int64_t wpr, int64_t nrows,
                                                  int64_t khalf, const int32_t* __restrict__ dst_ptr, int64_t n1,
                                                  int64_t n_in,
                                                  const int32_t* __restrict__ deg, const float* __restrict__ t,
                                                  int nfb, int64_t k, const float* __restrict__ b2,
                                                  const int32_t* __restrict__ ctl, const float* __restrict__ fef,
                                                  float* __restrict__ y) {
  const int64_t b = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (b >= nrows) return;
  const int cls = ctl[0];
  const float bias = b2 ? b2[cls] : 0.f;
  const uint64_t* mr = masks + b * wpr;
  const int32_t* dg = deg + b * n1;
  auto tval = [&](int64_t r, int64_t x) {
    float s = 0.f;
    for (int fb = 0; fb < nfb; ++fb) s += t[(static_cast<int64_t>(fb) * k + r) * n1 + x];
    return s;
  };
  {
    const float dv = __builtin_amdgcn_rsqf(1.0f + static_cast<float>(dg[0]));
    float acc = dv * tval(b, 0);
    bool live = false;
    for (int64_t x = 1; x < n_in; ++x) {
      const int64_t p = x - 1;
      if ((mr[p >> 6] >> (p & 63)) & 1) {
        live = true;
        acc = fmaf(__builtin_amdgcn_rsqf(1.0f + static_cast<float>(dg[x])), tval(b, x), acc);
      }
    }
    y[b] = live ? fmaf(dv, acc, bias) : fef[0];
  }
  if (PAIRS) {
    const int64_t bc = b + khalf;
    const float dv = __builtin_amdgcn_rsqf(1.0f + static_cast<float>((dst_ptr[1] - dst_ptr[0]) - dg[0]));
    float acc = dv * tval(bc, 0);
    bool live = false;
    for (int64_t x = 1; x < n_in; ++x) {
      const int64_t p = x - 1;
      if (!((mr[p >> 6] >> (p & 63)) & 1)) {
        live = true;
        const int nxx = dst_ptr[x + 1] - dst_ptr[x];
        acc = fmaf(__builtin_amdgcn_rsqf(1.0f + static_cast<float>(nxx - dg[x])), tval(bc, x), acc);
      }
    }
    y[bc] = live ? fmaf(dv, acc, bias) : fef[0];
  }
}

// Three layers on three hops, layer 2 at nodes 0 .. n2 - 1 (the target and
// its in-neighbours), whose in-neighbours all lie in H_1: by linearity of
// the transform, layer 2's sum at x is A W_2 with
//   A = d(x)^-1/2 H1[x] + sum_{e -> x, e in c} d(src e)^-1/2 H1[src e],
// so A is formed first (n2 rows per coalition instead of n1 for the
// transform).  The pass rows are the rows r0 .. r0 + nloc - 1 and, with
// pairs, their complements at pass rows nloc .. 2 nloc - 1 (mask bits and
// degrees complemented).  One workgroup per (node x, 16 pass rows): x's
// players are staged in LDS 256 at a time (source, players entering the
// source, and the 16 rows' mask bits of them); lane (rg, q) of wavefront w
// takes pass row 16 blk + 4 w + rg and features 4 q .. 4 q + 3 of each
// 64-feature chunk, four players' loads in flight.  Players in order, so
// the sums are the same in every call (an absent player adds 0).
constexpr int kAggRows = 16;
__global__ void __launch_bounds__(256) k_wide3_agg(const uint64_t* __restrict__ masks, int64_t wpr, int64_t r0,
                                                   int64_t nloc, bool pairs, const int32_t* __restrict__ dst_ptr,
                                                   const int32_t* __restrict__ edge_src, int64_t n1, int64_t n2,
                                                   const int32_t* __restrict__ deg, const float* __restrict__ H1,
                                                   int h, float* __restrict__ A) {
  __shared__ int32_t su[256], snu[256];
  __shared__ uint32_t sbits[kAggRows][8];   // each row's mask bits of the staged players (complemented rows: NOT)
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, rg = lane >> 4, q = lane & 15;
  const int64_t nr = pairs ? 2 * nloc : nloc;
  const int64_t x = blockIdx.x % n2;
  const int64_t lr0 = (blockIdx.x / n2) * kAggRows;
  // pass row lr -> (clamped pass row, complement?, contracted row)
  auto rowof = [&](int64_t lr, bool& comp, int64_t& row) {
    const int64_t lrc = lr < nr ? lr : nr - 1;
    comp = lrc >= nloc;
    row = r0 + (comp ? lrc - nloc : lrc);
    return lrc;
  };
  const int slot = 4 * wave + rg;
  const int64_t lr = lr0 + slot;
  const bool valid = lr < nr;
  bool comp;
  int64_t row;
  const int64_t lrc = rowof(lr, comp, row);
  const int32_t* dg = deg + row * n1;
  const float* hr = H1 + lrc * n1 * h;
  const int dgx = dg[x];
  const float dx = __builtin_amdgcn_rsqf(1.0f + static_cast<float>(comp ? (dst_ptr[x + 1] - dst_ptr[x]) - dgx : dgx));
  const int e0 = dst_ptr[x], e1 = dst_ptr[x + 1];
  const int64_t nbits = static_cast<int64_t>(wpr) * 64;   // bits of a mask row
  for (int f0 = 0; f0 < h; f0 += 64) {
    const int f = f0 + 4 * q;
    const bool fv = f < h;   // (h is a multiple of 16)
    const int fo = fv ? f : 0;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    {
      const float4 s4 = *reinterpret_cast<const float4*>(hr + x * h + fo);
      acc = make_float4(dx * s4.x, dx * s4.y, dx * s4.z, dx * s4.w);
    }
    for (int eb = e0; eb < e1; eb += 256) {
      const int n = e1 - eb < 256 ? e1 - eb : 256;
      __syncthreads();   // the previous chunk's reads are done
      if (tid < n) {
        const int32_t u = edge_src[eb + tid];
        su[tid] = u;
        snu[tid] = u < n1 ? dst_ptr[u + 1] - dst_ptr[u] : 0;
      }
      if (tid < kAggRows * 8) {
        // bits eb + 32 w .. + 31 of row slot tid / 8 (players past the chunk are never read)
        const int sl = tid >> 3, w = tid & 7;
        bool cs;
        int64_t rs;
        rowof(lr0 + sl, cs, rs);
        const int64_t pos = static_cast<int64_t>(eb) + 32 * w;
        uint32_t bits = 0;
        if (pos < nbits) {
          const uint64_t* mrs = masks + rs * wpr;
          const int64_t wi = pos >> 6;
          const int sh = static_cast<int>(pos & 63);
          const uint64_t lo = mrs[wi];
          const uint64_t hi = (sh > 32 && wi + 1 < wpr) ? mrs[wi + 1] : 0;
          bits = static_cast<uint32_t>(sh ? (lo >> sh) | (hi << (64 - sh)) : lo);
        }
        sbits[sl][w] = cs ? ~bits : bits;
      }
      __syncthreads();
      // four players at a time: absent players (coefficient 0) read x's own
      // row, already in the cache, so the four loads go out together
      for (int j0 = 0; j0 < n; j0 += 4) {
        int uq[4];
        bool pq[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const int j = j0 + t;
          const int jj = j < n ? j : 0;
          const int32_t u = su[jj];
          // (u >= n1 does not occur in an extracted subgraph: in-neighbours of these nodes lie in H_1)
          pq[t] = j < n && ((sbits[slot][jj >> 5] >> (jj & 31)) & 1u) && u < n1;
          uq[t] = pq[t] ? u : static_cast<int32_t>(x);
        }
        int dq[4];
        float4 vq[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          dq[t] = dg[uq[t]];
          vq[t] = *reinterpret_cast<const float4*>(hr + static_cast<int64_t>(uq[t]) * h + fo);
        }
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const int j = j0 + t < n ? j0 + t : 0;
          const int du = comp ? snu[j] - dq[t] : dq[t];
          const float c = pq[t] ? __builtin_amdgcn_rsqf(1.0f + static_cast<float>(du)) : 0.f;
          acc.x = fmaf(c, vq[t].x, acc.x);
          acc.y = fmaf(c, vq[t].y, acc.y);
          acc.z = fmaf(c, vq[t].z, acc.z);
          acc.w = fmaf(c, vq[t].w, acc.w);
        }
      }
    }
    if (valid && fv) *reinterpret_cast<float4*>(A + (lr * n2 + x) * h + f) = acc;
  }
}

// t[row][x] for nodes x < n2 from Z = A W_2 (rows as k_wide3_agg's):
// H2 = relu(d(x)^-1/2 Z + b_2), t = H2 . W_3[:, class]; one wavefront per
// (pass row, node), lane = feature, a fixed reduction order.
__global__ void __launch_bounds__(256) k_wide3_t(const uint64_t* __restrict__ masks, int64_t wpr, int64_t r0,
                                                 int64_t nloc, bool pairs, int64_t khalf,
                                                 const int32_t* __restrict__ dst_ptr, int64_t n1, int64_t n2,
                                                 const int32_t* __restrict__ deg, const float* __restrict__ Z, int h2,
                                                 const float* __restrict__ b2, const float* __restrict__ W3, int C,
                                                 const int32_t* __restrict__ ctl, int64_t k, float* __restrict__ t) {
  const int lane = threadIdx.x & 63;
  const int64_t item = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) >> 6;
  const int64_t nr = pairs ? 2 * nloc : nloc;
  if (item >= nr * n2) return;
  const int64_t lr = item / n2, x = item % n2;
  const bool comp = lr >= nloc;
  const int64_t row = r0 + (comp ? lr - nloc : lr);
  const int dgx = deg[row * n1 + x];
  const int d = comp ? (dst_ptr[x + 1] - dst_ptr[x]) - dgx : dgx;
  const float dx = __builtin_amdgcn_rsqf(1.0f + static_cast<float>(d));
  const int cls = ctl[0];
  const float* zr = Z + (lr * n2 + x) * h2;
  float s = 0.f;
  for (int f = lane; f < h2; f += 64) {
    const float hv = fmaxf(fmaf(dx, zr[f], b2 ? b2[f] : 0.f), 0.f);
    s = fmaf(hv, W3[static_cast<int64_t>(f) * C + cls], s);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
  if (lane == 0) t[(comp ? row + khalf : row) * n1 + x] = s;
}

// The two end coalitions (no players, every player), one layer, partial
// sums: Hp[p][x][f] = sum over part p of the players entering x (the 64
// wavefronts of the kEndParts workgroups of (x, feature block) take players
// w, w + 64, ...) of d(src)^-1/2 Z(src)[f] under E_c (degrees: the players
// entering each node); Z(u) = Zin[u] for u in H_1, Zc[u] otherwise (layer 1:
// both X W_1; layer 2 of a three-layer model: H^1 W_2 under E_c, and the
// constant rows); lane = feature, the sixteen wavefronts' sums added in a
// fixed order.  Nodes 0 .. nn - 1 (a prefix of H_1, one per blockIdx.x).
constexpr int kEndParts = 4;

__global__ void __launch_bounds__(1024) k_wide_ends_l1(const int32_t* __restrict__ dst_ptr,
                                                       const int32_t* __restrict__ edge_src, int64_t n1, int64_t nn,
                                                       const float* __restrict__ Zc, const float* __restrict__ Zin,
                                                       int h, float* __restrict__ Hp) {
  __shared__ float part[16][64];
  const int64_t x = blockIdx.x;
  const int pp = blockIdx.z;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int f = blockIdx.y * 64 + lane;
  const bool fv = f < h;
  const int e0 = dst_ptr[x], e1 = dst_ptr[x + 1];
  float acc = 0.f;
  for (int e = e0 + pp * 16 + wave; e < e1; e += 16 * kEndParts) {
    const int32_t u = edge_src[e];
    const float du = u < n1 ? __builtin_amdgcn_rsqf(1.0f + static_cast<float>(dst_ptr[u + 1] - dst_ptr[u])) : 1.0f;
    if (fv) acc = fmaf(du, (u < n1 ? Zin : Zc)[static_cast<int64_t>(u) * h + f], acc);
  }
  part[wave][lane] = acc;
  __syncthreads();
  if (wave == 0 && fv) {
    float a = 0.f;
    for (int i = 0; i < 16; ++i) a += part[i][lane];
    Hp[(static_cast<int64_t>(pp) * nn + x) * h + f] = a;
  }
}

// The end coalitions' layer at nodes 0 .. nn - 1 of H_1 from the parts' sums:
// Hf[x] under E_c (the sums in order, self loop Zself[x], bias, ReLU),
// Hf[nn] at the target under the empty coalition (its self loop only:
// Zempty, the target's input row then).  Then, with C > 0 (the last hidden
// layer; nodes 1 .. n_in - 1 are the target's in-neighbours, n_in <= nn),
// the output layer at the target for every class and the explained
// class (the requested one, or argmax f(E_c), ties to the lowest index):
// sp_y[c] = f_c(empty), sp_y[C + c] = f_c(E_c); ctl[0], class_out and
// f_empty_full as the other evaluation paths write them.  One workgroup of
// 1024 threads, one wavefront per class at a time (lane = feature).
__global__ void __launch_bounds__(1024) k_wide_ends_out(const int32_t* __restrict__ dst_ptr, int64_t nn,
                                                        int64_t n_in, const float* __restrict__ Hp,
                                                        const float* __restrict__ Zself,
                                                        const float* __restrict__ Zempty,
                                                        const float* __restrict__ b1, int h,
                                                        const float* __restrict__ W2, const float* __restrict__ b2,
                                                        int C, int requested, float* __restrict__ sp_y,
                                                        int32_t* __restrict__ ctl, int32_t* __restrict__ class_out,
                                                        float* __restrict__ f_empty_full, float* __restrict__ Hf) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int64_t i = threadIdx.x; i < nn * h; i += blockDim.x) {
    const int64_t x = i / h;
    const int f = static_cast<int>(i % h);
    float a = 0.f;
    for (int q = 0; q < kEndParts; ++q) a += Hp[(static_cast<int64_t>(q) * nn + x) * h + f];
    const float dx = __builtin_amdgcn_rsqf(1.0f + static_cast<float>(dst_ptr[x + 1] - dst_ptr[x]));
    const float bb = b1 ? b1[f] : 0.f;
    Hf[i] = fmaxf(fmaf(dx, fmaf(dx, Zself[x * h + f], a), bb), 0.f);
    if (x == 0) Hf[nn * h + f] = fmaxf(Zempty[f] + bb, 0.f);
  }
  if (C == 0) return;
  __syncthreads();
  const float dv = __builtin_amdgcn_rsqf(1.0f + static_cast<float>(dst_ptr[1] - dst_ptr[0]));
  for (int c = wave; c < C; c += 16) {
    float full = 0.f, empty = 0.f;
    for (int64_t x = 0; x < n_in; ++x) {
      float p = 0.f;
      for (int f = lane; f < h; f += 64) p = fmaf(Hf[x * h + f], W2[static_cast<int64_t>(f) * C + c], p);
      // node x >= 1 is the source of the target's player x - 1, present in E_c
      const float wx = x == 0 ? dv : __builtin_amdgcn_rsqf(1.0f + static_cast<float>(dst_ptr[x + 1] - dst_ptr[x]));
      full = fmaf(wx, p, full);
    }
    for (int f = lane; f < h; f += 64) empty = fmaf(Hf[nn * h + f], W2[static_cast<int64_t>(f) * C + c], empty);
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      full += __shfl_xor(full, off);
      empty += __shfl_xor(empty, off);
    }
    const float bb = b2 ? b2[c] : 0.f;
    if (lane == 0) {
      sp_y[c] = empty + bb;
      sp_y[C + c] = fmaf(dv, full, bb);
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int c = requested;
    if (c < 0) {
      c = 0;
      for (int i = 1; i < C; ++i)
        if (sp_y[C + i] > sp_y[C + c]) c = i;
    }
    ctl[0] = c;
    if (class_out) *class_out = c;
    f_empty_full[0] = sp_y[c];
    f_empty_full[1] = sp_y[C + c];
  }
}

}  // namespace

namespace gnnshap {

namespace {

bool wide_width(int h) { return h > 32 && h % 16 == 0 && h <= 4096; }

// Contracted rows per pass of a three-layer model: H1 and Z2 of a pass's
// rows and complements fill at most kPassBudget bytes, in whole 256-row
// blocks, and a pass has at least one block (so with thousands of nodes in
// H_1 the pass arrays exceed the budget).
constexpr int64_t kPassBudget = int64_t(1) << 30;

// Shared set-up: operand units and player lists, layer-1 operands and sums,
// degrees of the contracted rows.
int wide_prep(const WideShape& s, const WideWs& w, const gnnshap_subgraph* sg, const uint64_t* masks, int64_t wpr,
              const float* Zc, bool pairs, hipStream_t st) {
  if (pairs && (s.k & 1)) return fail(GNNSHAP_EINVAL, "complement pairs need an even number of rows");
  if (s.n1 > INT32_MAX / 2 || s.M > INT32_MAX / 2) return fail(GNNSHAP_EUNSUPPORTED, "subgraph too large");
  const int64_t nrows = pairs ? s.k / 2 : s.k;
  k_wide_prep<<<1, 1024, 0, st>>>(sg->dst_ptr, sg->edge_src, s.n1, w.seg, w.spec_ptr, w.spec_e);
  GS_LAUNCHED();
  k_wide_zop<<<grid_for(s.units_cap * s.ntot * 64, 256, 16384), 256, 0, st>>>(
      sg->dst_ptr, sg->edge_src, s.n1, s.n1, w.seg, Zc, s.h, s.ntot, s.units_cap, w.Zop);
  GS_LAUNCHED();
  if (pairs) {
    k_wide_sum<<<static_cast<unsigned>(s.n1 * s.ntot), 1024, 0, st>>>(sg->dst_ptr, sg->edge_src, s.n1, Zc, s.h,
                                                                      s.ntot, w.S);
    GS_LAUNCHED();
  }
  k_wide_deg<<<grid_for(nrows * s.n1, 256, 16384), 256, 0, st>>>(masks, wpr, nrows, sg->dst_ptr, s.n1, w.deg);
  GS_LAUNCHED();
  return GNNSHAP_OK;
}

// One contraction launch over the pass r0 .. r0 + nloc - 1 at nodes
// 0 .. nx - 1 of H_1 (see k_wide_l1).
template <int MODE>
int wide_layer(const WideShape& s, const gnnshap_subgraph* sg, const uint64_t* masks, int64_t wpr, int64_t r0,
               int64_t nloc, int64_t nx, bool pairs, const uint4* Zop, int ntot, int nfb, int h, const float* Zc,
               const float* S, const WideWs& w, const float* b, const float* Wp, const int32_t* ctl,
               const float* Zrow, float* Hout, hipStream_t st) {
  if (nloc <= 0) return GNNSHAP_OK;
  const int64_t khalf = pairs ? s.k / 2 : 0;
  const int64_t cblocks = ceil_div(nloc, kBlockRows);
  if (nx * cblocks > INT32_MAX || nfb > 65535) return fail(GNNSHAP_EUNSUPPORTED, "evaluation grid too large");
  const dim3 grid(static_cast<unsigned>(nx * cblocks), static_cast<unsigned>(nfb));
  if (pairs)
    k_wide_l1<true, MODE><<<grid, kBlockRows, 0, st>>>(masks, wpr, r0, nloc, khalf, cblocks, sg->dst_ptr,
                                                       sg->edge_src, s.n1, w.seg, Zop, ntot, h, Zc, S, w.spec_ptr,
                                                       w.spec_e, w.deg, b, Wp, s.C, ctl, w.t, s.k, Zrow, Hout);
  else
    k_wide_l1<false, MODE><<<grid, kBlockRows, 0, st>>>(masks, wpr, r0, nloc, khalf, cblocks, sg->dst_ptr,
                                                        sg->edge_src, s.n1, w.seg, Zop, ntot, h, Zc, S, w.spec_ptr,
                                                        w.spec_e, w.deg, b, Wp, s.C, ctl, w.t, s.k, Zrow, Hout);
  GS_LAUNCHED();
  return GNNSHAP_OK;
}

int wide_out(const WideShape& s, const WideWs& w, const gnnshap_subgraph* sg, const uint64_t* masks, int64_t wpr,
             int nfb_t, const float* b_last, const int32_t* ctl, const float* fef, bool pairs, float* y,
             hipStream_t st) {
  const int64_t nrows = pairs ? s.k / 2 : s.k;
  const int64_t khalf = pairs ? s.k / 2 : 0;
  const unsigned g = static_cast<unsigned>(ceil_div(nrows, 256));
  GS_TIMED("k_wide_out", st);
  if (pairs)
    k_wide_out<true><<<g, 256, 0, st>>>(masks, wpr, nrows, khalf, sg->dst_ptr, s.n1, s.n2, w.deg, w.t, nfb_t, s.k,
                                        b_last, ctl, fef, y);
  else
    k_wide_out<false><<<g, 256, 0, st>>>(masks, wpr, nrows, khalf, sg->dst_ptr, s.n1, s.n2, w.deg, w.t, nfb_t, s.k,
                                         b_last, ctl, fef, y);
  GS_LAUNCHED();
  return GNNSHAP_OK;
}

}  // namespace

bool wide_applies(int num_layers, int num_hops, const int32_t* dims) {
  const bool shape = (num_hops == 2 && (num_layers == 2 || num_layers == 3)) || (num_hops == 3 && num_layers == 3);
  if (!shape) return false;
  for (int j = 1; j < num_layers; ++j)
    if (!wide_width(dims[j])) return false;
  return true;
}

WideShape wide_shape(int64_t M, int64_t n_nodes, int64_t n1, int64_t n2, int64_t k, const int32_t* dims,
                     int num_layers) {
  WideShape s;
  s.M = M;
  s.n_nodes = n_nodes;
  s.n1 = n1;
  s.n2 = n2;
  s.k = k;
  s.h = dims[1];
  s.C = dims[num_layers];
  s.ntot = s.h / 16;
  s.nfb = static_cast<int>(ceil_div(s.ntot, kTiles));
  s.units_cap = ceil_div(M, kUnit) + n1;
  if (num_layers == 3) {
    s.h2 = dims[2];
    s.ntot2 = s.h2 / 16;
    s.nfb2 = static_cast<int>(ceil_div(s.ntot2, kTiles));
    s.agg3 = n2 < n1;
    const int64_t per_row = 2 * (n1 * (static_cast<int64_t>(s.h) + s.h2) + (s.agg3 ? n2 * s.h : 0)) *
                            static_cast<int64_t>(sizeof(float));
    int64_t p = kPassBudget / per_row;
    p = std::max<int64_t>(kBlockRows, p - p % kBlockRows);
    s.pass = std::min<int64_t>(p, k);
  }
  return s;
}

WideWs wide_carve(Carver& c, const WideShape& s) {
  WideWs w{};
  w.seg = c.take<int32_t>(s.n1 + 1);
  w.spec_ptr = c.take<int32_t>(s.n1 + 1);
  w.spec_e = c.take<int32_t>(s.M);
  w.Zop = c.take<uint4>(s.units_cap * s.ntot * kParts * 64);
  w.S = c.take<float>(s.n1 * s.h);
  w.deg = c.take<int32_t>(s.k * s.n1);
  w.t = c.take<float>(static_cast<int64_t>(s.h2 ? (s.agg3 ? 1 : s.nfb2) : s.nfb) * s.k * s.n1);
  w.hf = c.take<float>((s.n1 + 1) * s.h);
  w.hp = c.take<float>(kEndParts * s.n1 * std::max(s.h, s.h2));
  if (s.h2 > 0) {
    w.z2e = c.take<float>((s.n1 + 1) * s.h2);
    w.hf2 = c.take<float>((s.n1 + 1) * s.h2);
    w.Zop2 = c.take<uint4>(s.units_cap * s.ntot2 * kParts * 64);
    w.S2 = c.take<float>(s.n1 * s.h2);
    w.H1 = c.take<float>(2 * s.pass * s.n1 * s.h);
    w.Z2 = c.take<float>(2 * s.pass * s.n1 * s.h2);
    w.A3 = s.agg3 ? c.take<float>(2 * s.pass * s.n2 * s.h) : nullptr;
  }
  return w;
}

int launch_wide_ends(const WideShape& s, const WideWs& w, const gnnshap_subgraph* sg, const float* Zc, const float* b1,
                     const float* W2, const float* b2, int32_t target_class, float* sp_y, int32_t* ctl,
                     int32_t* class_out, float* f_empty_full, hipStream_t st) {
  if (s.n1 > 65535 * 64) return fail(GNNSHAP_EUNSUPPORTED, "too many nodes in H_1");
  {
    GS_TIMED("k_wide_ends", st);
    k_wide_ends_l1<<<dim3(static_cast<unsigned>(s.n1), static_cast<unsigned>(ceil_div(s.h, 64)), kEndParts), 1024, 0,
                     st>>>(sg->dst_ptr, sg->edge_src, s.n1, s.n1, Zc, Zc, s.h, w.hp);
    GS_LAUNCHED();
    k_wide_ends_out<<<1, 1024, 0, st>>>(sg->dst_ptr, s.n1, s.n2, w.hp, Zc, Zc, b1, s.h, W2, b2, s.C, target_class,
                                         sp_y, ctl, class_out, f_empty_full, w.hf);
  }
  GS_LAUNCHED();
  return GNNSHAP_OK;
}

int launch_wide(const WideShape& s, const WideWs& w, const gnnshap_subgraph* sg, const uint64_t* masks, int64_t wpr,
                const float* Zc, const float* b1, const float* W2, const float* b2, const int32_t* ctl,
                const float* fef, bool pairs, float* y, hipStream_t st) {
  if (int r = wide_prep(s, w, sg, masks, wpr, Zc, pairs, st)) return r;
  {
    GS_TIMED("k_wide_l1", st);
    if (int r = wide_layer<kProj>(s, sg, masks, wpr, 0, pairs ? s.k / 2 : s.k, s.n1, pairs, w.Zop, s.ntot, s.nfb, s.h,
                                  Zc, w.S, w, b1, W2, ctl, nullptr, nullptr, st))
      return r;
  }
  return wide_out(s, w, sg, masks, wpr, s.nfb, b2, ctl, fef, pairs, y, st);
}

int launch_wide3_ends_l1(const WideShape& s, const WideWs& w, const gnnshap_subgraph* sg, const float* Zc1,
                         const float* b1, hipStream_t st) {
  if (s.h2 == 0) return fail(GNNSHAP_EINVAL, "not a three-layer shape");
  if (s.n1 > 65535 * 64) return fail(GNNSHAP_EUNSUPPORTED, "too many nodes in H_1");
  GS_TIMED("k_wide_ends", st);
  k_wide_ends_l1<<<dim3(static_cast<unsigned>(s.n1), static_cast<unsigned>(ceil_div(s.h, 64)), kEndParts), 1024, 0,
                   st>>>(sg->dst_ptr, sg->edge_src, s.n1, s.n1, Zc1, Zc1, s.h, w.hp);
  GS_LAUNCHED();
  k_wide_ends_out<<<1, 1024, 0, st>>>(sg->dst_ptr, s.n1, s.n2, w.hp, Zc1, Zc1, b1, s.h, nullptr, nullptr, 0, -1,
                                       nullptr, nullptr, nullptr, nullptr, w.hf);
  GS_LAUNCHED();
  return GNNSHAP_OK;
}

int launch_wide3_ends_l2(const WideShape& s, const WideWs& w, const gnnshap_subgraph* sg, const float* Zc2,
                         const float* b2, const float* W3, const float* b3, int32_t target_class, float* sp_y,
                         int32_t* ctl, int32_t* class_out, float* f_empty_full, hipStream_t st) {
  if (s.h2 == 0) return fail(GNNSHAP_EINVAL, "not a three-layer shape");
  GS_TIMED("k_wide_ends", st);
  // layer 2 is needed at the target and its in-neighbours only (nodes 0 .. n2 - 1)
  k_wide_ends_l1<<<dim3(static_cast<unsigned>(s.n2), static_cast<unsigned>(ceil_div(s.h2, 64)), kEndParts), 1024, 0,
                   st>>>(sg->dst_ptr, sg->edge_src, s.n1, s.n2, Zc2, w.z2e, s.h2, w.hp);
  GS_LAUNCHED();
  k_wide_ends_out<<<1, 1024, 0, st>>>(sg->dst_ptr, s.n2, s.n2, w.hp, w.z2e, w.z2e + s.n1 * s.h2, b2, s.h2, W3, b3,
                                       s.C, target_class, sp_y, ctl, class_out, f_empty_full, w.hf2);
  GS_LAUNCHED();
  return GNNSHAP_OK;
}

int launch_wide3_prep(const WideShape& s, const WideWs& w, const gnnshap_subgraph* sg, const uint64_t* masks,
                      int64_t wpr, const float* Zc1, const float* Zc2, bool pairs, hipStream_t st) {
  if (s.h2 == 0) return fail(GNNSHAP_EINVAL, "not a three-layer shape");
  if (int r = wide_prep(s, w, sg, masks, wpr, Zc1, pairs, st)) return r;
  if (s.agg3) return GNNSHAP_OK;   // layer 2 from A W_2 (no contraction)
  // layer 2's operands at nodes 0 .. n2 - 1 (where layer 2 is needed): the
  // input rows of the sources outside H_1 (their degree is 1 under every
  // coalition, so the rows are constant)
  k_wide_zop<<<grid_for(s.units_cap * s.ntot2 * 64, 256, 16384), 256, 0, st>>>(
      sg->dst_ptr, sg->edge_src, s.n1, s.n2, w.seg, Zc2, s.h2, s.ntot2, s.units_cap, w.Zop2);
  GS_LAUNCHED();
  if (pairs) {
    k_wide_sum<<<static_cast<unsigned>(s.n2 * s.ntot2), 1024, 0, st>>>(sg->dst_ptr, sg->edge_src, s.n1, Zc2, s.h2,
                                                                       s.ntot2, w.S2);
    GS_LAUNCHED();
  }
  return GNNSHAP_OK;
}

int launch_wide3_l1(const WideShape& s, const WideWs& w, const gnnshap_subgraph* sg, const uint64_t* masks,
                    int64_t wpr, int64_t r0, int64_t nloc, const float* Zc1, const float* b1, bool pairs,
                    hipStream_t st) {
  if (nloc > s.pass) return fail(GNNSHAP_EINVAL, "pass larger than the workspace's");
  GS_TIMED("k_wide_l1", st);
  return wide_layer<kFull>(s, sg, masks, wpr, r0, nloc, s.n1, pairs, w.Zop, s.ntot, s.nfb, s.h, Zc1, w.S, w, b1,
                           nullptr, nullptr, nullptr, w.H1, st);
}

int launch_wide3_l2(const WideShape& s, const WideWs& w, const gnnshap_subgraph* sg, const uint64_t* masks,
                    int64_t wpr, int64_t r0, int64_t nloc, const float* b2, const float* W3, const int32_t* ctl,
                    bool pairs, hipStream_t st) {
  if (nloc > s.pass) return fail(GNNSHAP_EINVAL, "pass larger than the workspace's");
  GS_TIMED("k_wide_l2", st);
  return wide_layer<kProjRows>(s, sg, masks, wpr, r0, nloc, s.n2, pairs, w.Zop2, s.ntot2, s.nfb2, s.h2, nullptr,
                               w.S2, w, b2, W3, ctl, w.Z2, nullptr, st);
}

int launch_wide3_agg(const WideShape& s, const WideWs& w, const gnnshap_subgraph* sg, const uint64_t* masks,
                     int64_t wpr, int64_t r0, int64_t nloc, bool pairs, hipStream_t st) {
  if (nloc > s.pass) return fail(GNNSHAP_EINVAL, "pass larger than the workspace's");
  if (nloc <= 0) return GNNSHAP_OK;
  const int64_t blocks = ceil_div((pairs ? 2 : 1) * nloc, kAggRows) * s.n2;
  if (blocks > INT32_MAX) return fail(GNNSHAP_EUNSUPPORTED, "evaluation grid too large");
  GS_TIMED("k_wide3_agg", st);
  k_wide3_agg<<<static_cast<unsigned>(blocks), 256, 0, st>>>(
      masks, wpr, r0, nloc, pairs, sg->dst_ptr, sg->edge_src, s.n1, s.n2, w.deg, w.H1, s.h, w.A3);
  GS_LAUNCHED();
  return GNNSHAP_OK;
}

int launch_wide3_t(const WideShape& s, const WideWs& w, const gnnshap_subgraph* sg, const uint64_t* masks,
                   int64_t wpr, int64_t r0, int64_t nloc, const float* b2, const float* W3, const int32_t* ctl,
                   bool pairs, hipStream_t st) {
  if (nloc > s.pass) return fail(GNNSHAP_EINVAL, "pass larger than the workspace's");
  if (nloc <= 0) return GNNSHAP_OK;
  const int64_t items = (pairs ? 2 : 1) * nloc * s.n2;
  if (ceil_div(items * 64, 256) > INT32_MAX) return fail(GNNSHAP_EUNSUPPORTED, "evaluation grid too large");
  k_wide3_t<<<static_cast<unsigned>(ceil_div(items * 64, 256)), 256, 0, st>>>(
      masks, wpr, r0, nloc, pairs, pairs ? s.k / 2 : 0, sg->dst_ptr, s.n1, s.n2, w.deg, w.Z2, s.h2, b2, W3, s.C, ctl,
      s.k, w.t);
  GS_LAUNCHED();
  return GNNSHAP_OK;
}

int launch_wide3_out(const WideShape& s, const WideWs& w, const gnnshap_subgraph* sg, const uint64_t* masks,
                     int64_t wpr, const float* b3, const int32_t* ctl, const float* fef, bool pairs, float* y,
                     hipStream_t st) {
  return wide_out(s, w, sg, masks, wpr, s.agg3 ? 1 : s.nfb2, b3, ctl, fef, pairs, y, st);
}

}  // namespace gnnshap
