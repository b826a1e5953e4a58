// Host-side sample plan (Sec. 3.3.1, eq. 4-6, Alg. 2 of the GNNShap paper).
//
// Every floating-point operation is fp64, in a fixed order (plain ascending
// sums, no fused multiply-add: this file is compiled with -ffp-contract=off),
// so the plan is reproducible bit for bit on any IEEE-754 host.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <vector>

#include "gnnshap.h"

namespace gnnshap {
int fail(int status, const char* fmt, ...);
void clear_error();
}  // namespace gnnshap

namespace {

constexpr int64_t kSaturate = int64_t(1) << 62;
constexpr int64_t kMaxRows = int64_t(1) << 31;

// C(n, r) saturated at 2^62: C(n-r+i, i) = C(n-r+i-1, i-1) (n-r+i) / i is an
// exact integer at every step.
int64_t binom_sat(int64_t n, int64_t r) {
  if (r < 0 || r > n) return 0;
  r = std::min(r, n - r);
  unsigned __int128 v = 1;
  for (int64_t i = 1; i <= r; ++i) {
    v = v * static_cast<unsigned __int128>(n - r + i) / static_cast<unsigned __int128>(i);
    if (v >= static_cast<unsigned __int128>(kSaturate)) return kSaturate;
  }
  return static_cast<int64_t>(v);
}

double ascending_sum(const std::vector<double>& v, size_t from, size_t to) {
  double s = 0.0;
  for (size_t i = from; i < to; ++i) s = s + v[i];
  return s;
}

}  // namespace

extern "C" int gnnshap_plan_samples(gnnshap_sample_plan* plan, gnnshap_class* classes,
                                    int64_t cap_classes) {
  try {
    gnnshap::clear_error();
    if (!plan) return gnnshap::fail(GNNSHAP_EINVAL, "plan is NULL");
    const int64_t M = plan->num_players;
    const int64_t p = plan->num_samples;
    if (M < 2) return gnnshap::fail(GNNSHAP_EINVAL, "need at least 2 players (M=%lld)", (long long)M);
    if (p < 2 || (p % 2) != 0)
      return gnnshap::fail(GNNSHAP_EINVAL, "sample budget must be even and >= 2 (p=%lld)", (long long)p);
    if (M > (int64_t(1) << 30)) return gnnshap::fail(GNNSHAP_EINVAL, "too many players");

    // Size classes c = 1..M/2 (eq. 4): omega_c = kappa_c * rho_c.
    const int64_t K = M / 2;
    std::vector<double> omega(K);
    std::vector<int64_t> ncoal(K);
    for (int64_t c = 1; c <= K; ++c) {
      const bool paired = 2 * c < M;
      const double kappa = paired ? 2.0 : 1.0;
      const double rho = static_cast<double>(M - 1) / (static_cast<double>(c) * static_cast<double>(M - c));
      omega[c - 1] = kappa * rho;
      int64_t n = binom_sat(M, c);
      if (!paired && n < kSaturate) n /= 2;
      ncoal[c - 1] = n;
    }
    const double omega_total = ascending_sum(omega, 0, K);

    // Surplus redistribution: enumerate classes whose eq. 5 share covers them.
    int64_t pairs = p / 2;
    int64_t n_full = 0;
    for (int64_t i = 0; i < K; ++i) {
      const double w_rem = ascending_sum(omega, i, K);
      const double share = (static_cast<double>(pairs) * omega[i]) / w_rem;
      if (ncoal[i] <= pairs && static_cast<double>(ncoal[i]) <= share + 1e-6) {
        ++n_full;
        pairs -= ncoal[i];
      } else {
        break;
      }
    }

    // Largest-remainder bins for the random classes (eq. 5).
    std::vector<int64_t> bins(K, 0);
    int64_t p_r = 0;
    if (n_full < K) {
      p_r = pairs;
      const double w_r = ascending_sum(omega, n_full, K);
      std::vector<double> frac(K, 0.0);
      int64_t assigned = 0;
      for (int64_t i = n_full; i < K; ++i) {
        const double q = (static_cast<double>(p_r) * omega[i]) / w_r;
        bins[i] = static_cast<int64_t>(std::floor(q));
        frac[i] = q - static_cast<double>(bins[i]);
        assigned += bins[i];
      }
      std::vector<int64_t> order;
      order.reserve(K - n_full);
      for (int64_t i = n_full; i < K; ++i) order.push_back(i);
      std::sort(order.begin(), order.end(), [&](int64_t a, int64_t b) {
        if (frac[a] != frac[b]) return frac[a] > frac[b];
        return a < b;
      });
      const int64_t extra = p_r - assigned;
      for (int64_t t = 0; t < extra; ++t) bins[order[t]] += 1;
    }

    // Row layout and weights.
    int64_t n_classes = n_full;
    for (int64_t i = n_full; i < K; ++i) n_classes += bins[i] > 0 ? 1 : 0;
    int64_t half = 0;
    for (int64_t i = 0; i < n_full; ++i) half += ncoal[i];
    half += p_r;
    if (2 * half > kMaxRows) return gnnshap::fail(GNNSHAP_EINVAL, "more than 2^31 rows");

    double full_fraction = 0.0;
    std::vector<gnnshap_class> out;
    out.reserve(n_classes);
    int64_t row = 0;
    for (int64_t i = 0; i < n_full; ++i) {
      const double f = omega[i] / omega_total;
      full_fraction = full_fraction + f;
      gnnshap_class cl;
      cl.size = static_cast<int32_t>(i + 1);
      cl.full = 1;
      cl.row_begin = row;
      cl.row_count = ncoal[i];
      cl.weight = f / (2.0 * static_cast<double>(ncoal[i]));
      out.push_back(cl);
      row += ncoal[i];
    }
    const int64_t random_begin = row;
    const double random_weight =
        p_r > 0 ? (1.0 - full_fraction) / (2.0 * static_cast<double>(p_r)) : 0.0;
    for (int64_t i = n_full; i < K; ++i) {
      if (bins[i] == 0) continue;
      gnnshap_class cl;
      cl.size = static_cast<int32_t>(i + 1);
      cl.full = 0;
      cl.row_begin = row;
      cl.row_count = bins[i];
      cl.weight = random_weight;
      out.push_back(cl);
      row += bins[i];
    }

    plan->num_rows = 2 * half;
    plan->words_per_row = (M + 63) / 64;
    plan->num_classes = n_classes;
    plan->random_begin = random_begin;
    plan->full_fraction = full_fraction;
    plan->random_weight = random_weight;
    if (!classes || cap_classes < n_classes)
      return gnnshap::fail(GNNSHAP_ECAPACITY, "class table needs %lld records", (long long)n_classes);
    std::copy(out.begin(), out.end(), classes);
    return GNNSHAP_OK;
  } catch (...) {
    return gnnshap::fail(GNNSHAP_EHIP, "unexpected C++ exception in plan");
  }
}
