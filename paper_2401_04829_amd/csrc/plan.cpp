// Host-side sample plan (Sec. 3.3.1, eq. 4-6, Alg. 2 of the GNNShap paper).
//
// Every floating-point operation is fp64, in a fixed order (plain ascending
// sums, no fused multiply-add: this file is compiled with -ffp-contract=off),
// so the plan is reproducible bit for bit on any IEEE-754 host.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <memory>
#include <mutex>
#include <string>
#include <unordered_map>
#include <utility>
#include <vector>

#include "gnnshap.h"

namespace gnnshap {
int fail(int status, const char* fmt, ...);
void clear_error();
}  // namespace gnnshap

namespace {

constexpr int64_t kSaturate = int64_t(1) << 62;
constexpr int64_t kMaxRows = int64_t(1) << 31;

// C(M, c) for c = 1 .. K, saturated at 2^62, by the recurrence
// C(M, c) = C(M, c-1) (M-c+1) / c (exact in integers at every step; the
// sequence grows up to c = M/2, so it stays saturated once it saturates).
void binom_row(int64_t M, int64_t K, std::vector<int64_t>& out) {
  unsigned __int128 v = 1;
  bool sat = false;
  for (int64_t c = 1; c <= K; ++c) {
    if (!sat) {
      v = v * static_cast<unsigned __int128>(M - c + 1) / static_cast<unsigned __int128>(c);
      sat = v >= static_cast<unsigned __int128>(kSaturate);
    }
    out[c - 1] = sat ? kSaturate : static_cast<int64_t>(v);
  }
}

double ascending_sum(const std::vector<double>& v, size_t from, size_t to) {
  double s = 0.0;
  for (size_t i = from; i < to; ++i) s = s + v[i];
  return s;
}

// Eq. 4-6 and Alg. 2 for one (M, p): fills the outputs of *plan and `out`.
int plan_one(gnnshap_sample_plan* plan, std::vector<gnnshap_class>& out) {
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
  binom_row(M, K, ncoal);
  for (int64_t c = 1; c <= K; ++c) {
    const bool paired = 2 * c < M;
    const double kappa = paired ? 2.0 : 1.0;
    const double rho = static_cast<double>(M - 1) / (static_cast<double>(c) * static_cast<double>(M - c));
    omega[c - 1] = kappa * rho;
    if (!paired && ncoal[c - 1] < kSaturate) ncoal[c - 1] /= 2;
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
  int64_t half = 0;
  for (int64_t i = 0; i < n_full; ++i) half += ncoal[i];
  half += p_r;
  if (2 * half > kMaxRows) return gnnshap::fail(GNNSHAP_EINVAL, "more than 2^31 rows");

  double full_fraction = 0.0;
  out.clear();
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
  plan->num_classes = static_cast<int64_t>(out.size());
  plan->random_begin = random_begin;
  plan->full_fraction = full_fraction;
  plan->random_weight = random_weight;
  return GNNSHAP_OK;
}

// Plans depend on (M, p) only; serving loops ask for the same sizes again
// and again, so computed plans are kept (at most kCacheEntries, then the
// cache starts over).  Lookups and inserts hold one mutex.
constexpr size_t kCacheEntries = 4096;

struct Planned {
  gnnshap_sample_plan plan;
  std::vector<gnnshap_class> classes;
};

struct PairHash {
  size_t operator()(const std::pair<int64_t, int64_t>& k) const {
    return std::hash<int64_t>()(k.first * 1000003 + k.second);
  }
};

std::mutex g_cache_mu;
std::unordered_map<std::pair<int64_t, int64_t>, std::shared_ptr<const Planned>, PairHash> g_cache;

// The plan of (M, p) into *out, computed or from the cache.
int planned(int64_t M, int64_t p, std::shared_ptr<const Planned>* out) {
  const std::pair<int64_t, int64_t> key(M, p);
  {
    std::lock_guard<std::mutex> lock(g_cache_mu);
    auto it = g_cache.find(key);
    if (it != g_cache.end()) {
      *out = it->second;
      return GNNSHAP_OK;
    }
  }
  auto e = std::make_shared<Planned>();
  e->plan = gnnshap_sample_plan{};
  e->plan.num_players = M;
  e->plan.num_samples = p;
  if (int st = plan_one(&e->plan, e->classes)) return st;
  std::lock_guard<std::mutex> lock(g_cache_mu);
  if (g_cache.size() >= kCacheEntries) g_cache.clear();
  g_cache.emplace(key, e);
  *out = e;
  return GNNSHAP_OK;
}

}  // namespace

extern "C" int gnnshap_plan_samples(gnnshap_sample_plan* plan, gnnshap_class* classes,
                                    int64_t cap_classes) {
  try {
    gnnshap::clear_error();
    if (!plan) return gnnshap::fail(GNNSHAP_EINVAL, "plan is NULL");
    std::shared_ptr<const Planned> e;
    if (int st = planned(plan->num_players, plan->num_samples, &e)) return st;
    const uint64_t seed = plan->seed, stream_id = plan->stream_id;
    const int64_t threshold = plan->iterative_threshold;
    *plan = e->plan;
    plan->seed = seed;
    plan->stream_id = stream_id;
    plan->iterative_threshold = threshold;
    if (!classes || cap_classes < plan->num_classes)
      return gnnshap::fail(GNNSHAP_ECAPACITY, "class table needs %lld records", (long long)plan->num_classes);
    std::copy(e->classes.begin(), e->classes.end(), classes);
    return GNNSHAP_OK;
  } catch (...) {
    return gnnshap::fail(GNNSHAP_EHIP, "unexpected C++ exception in plan");
  }
}

extern "C" int gnnshap_plan_batch(const gnnshap_subgraph* sgs, const int64_t* stream_ids, int64_t n,
                                  int64_t num_samples, uint64_t seed, gnnshap_sample_plan* plans,
                                  gnnshap_class* classes, int64_t cap_classes, int64_t* num_classes,
                                  int64_t* totals) {
  try {
    gnnshap::clear_error();
    if (!sgs || !stream_ids || !plans || !num_classes) return gnnshap::fail(GNNSHAP_EINVAL, "null argument");
    if (n < 1) return gnnshap::fail(GNNSHAP_EINVAL, "need at least one target");
    int64_t ncls = 0, words = 0, rows = 0, players = 0;
    for (int64_t t = 0; t < n; ++t) {
      const int64_t M = sgs[t].num_edges;
      std::shared_ptr<const Planned> e;
      if (int st = planned(M, num_samples, &e)) {
        const std::string why = gnnshap_last_error();
        return gnnshap::fail(st, "target %lld: %s", (long long)t, why.c_str());
      }
      gnnshap_sample_plan& pt = plans[t];
      pt = e->plan;
      pt.seed = seed;
      pt.stream_id = static_cast<uint64_t>(stream_ids[t]);
      pt.iterative_threshold = 0;
      if (classes && ncls + pt.num_classes <= cap_classes)
        std::copy(e->classes.begin(), e->classes.end(), classes + ncls);
      ncls += pt.num_classes;
      words += pt.num_rows * pt.words_per_row;
      rows += pt.num_rows;
      players += M;
    }
    *num_classes = ncls;
    if (totals) {
      totals[0] = words;
      totals[1] = rows;
      totals[2] = players;
    }
    if (!classes || cap_classes < ncls)
      return gnnshap::fail(GNNSHAP_ECAPACITY, "class tables need %lld records", (long long)ncls);
    return GNNSHAP_OK;
  } catch (...) {
    return gnnshap::fail(GNNSHAP_EHIP, "unexpected C++ exception in plan");
  }
}
