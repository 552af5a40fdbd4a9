// KV-cache pool planner (Section 3.1, "KV-cache Planner and Virtualizer";
// Eq. 1-2): the pool page budget as a high quantile of the aggregate active
// KV bytes at a random observation time, by trace-driven Monte Carlo.
//
// Request i of model M arrives at A_i with O_p,i prompt tokens, O_d,i output
// tokens and decode residence time T_i. At age u its active KV grows
// linearly from O_p,i to O_p,i + O_d,i over [0, T_i) and is released at T_i
// (Eq. 1); the pool demand at time t sums kappa(M) times the active tokens of
// every request of every model (Eq. 2). Each simulated arrival draws one
// whole trace record, which keeps the empirical correlations between prompt
// length, output length and residence time.
//
// The procedure where the paper leaves it open: Poisson arrivals of rate
// lambda_M per model over [0, H); observation times uniform over [W, H)
// with W the longest residence time; the q-quantile is the order statistic
// of rank ceil(q n); the budget rounds it up to whole allocator chunks.
// Random draws come from SplitMix64 (Steele, Lea and Flood, OOPSLA 2014),
// one stream from the caller's seed: per model in order, an inter-arrival
// uniform then a record uniform until an arrival falls at or past H (whose
// record uniform is not drawn), then the observation uniforms.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <vector>

#include "crosspool.h"
#include "status.hpp"

namespace {

struct SplitMix64 {
  uint64_t state;
  uint64_t next() {
    state += 0x9E3779B97F4A7C15ull;
    uint64_t z = state;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
  }
  double uniform() { return (double)(next() >> 11) * (1.0 / 9007199254740992.0); }
};

struct Arrival {
  double a, kappa, op, od, tr;
};

}  // namespace

extern "C" {

cp_status cp_plan_pool(const cp_plan_model *models, int32_t n_models, const cp_plan_opts *opts,
                       cp_plan_result *out) {
  using cp::fail;
  if (!models || n_models < 1) return fail(CP_EINVAL, "no models to plan for");
  if (!opts || !out) return fail(CP_EINVAL, "null opts or result");
  const double H = opts->horizon_s, q = opts->quantile;
  if (!(H > 0) || !std::isfinite(H)) return fail(CP_EINVAL, "horizon must be positive and finite");
  if (!(q > 0 && q <= 1)) return fail(CP_EINVAL, "quantile must lie in (0, 1]");
  if (opts->n_obs < 1) return fail(CP_EINVAL, "at least one observation");
  if (opts->chunk_bytes == 0) return fail(CP_EINVAL, "chunk_bytes must be positive");
  double W = 0;
  for (int32_t m = 0; m < n_models; ++m) {
    const cp_plan_model &d = models[m];
    if (d.n_samples < 1 || !d.prompt_tokens || !d.output_tokens || !d.service_time_s)
      return fail(CP_EINVAL, "model %d: no trace samples", m);
    if (!(d.kappa_bytes > 0) || !(d.arrival_rate > 0) || !std::isfinite(d.arrival_rate))
      return fail(CP_EINVAL, "model %d: kappa and arrival rate must be positive", m);
    for (int64_t j = 0; j < d.n_samples; ++j) {
      if (d.prompt_tokens[j] < 0 || d.output_tokens[j] < 0)
        return fail(CP_EINVAL, "model %d, record %lld: negative token count", m, (long long)j);
      if (!(d.service_time_s[j] > 0) || !std::isfinite(d.service_time_s[j]))
        return fail(CP_EINVAL, "model %d, record %lld: residence time must be positive", m, (long long)j);
      W = std::max(W, d.service_time_s[j]);
    }
    if (d.arrival_rate * H > 1e8) return fail(CP_EINVAL, "model %d: more than 1e8 expected arrivals", m);
  }
  if (!(H > W)) return fail(CP_EINVAL, "the horizon must exceed the longest residence time");

  SplitMix64 rng{opts->seed};
  std::vector<Arrival> arr;
  for (int32_t m = 0; m < n_models; ++m) {
    const cp_plan_model &d = models[m];
    double t = 0;
    for (;;) {
      t += -std::log1p(-rng.uniform()) / d.arrival_rate;
      if (t >= H) break;
      const int64_t j = std::min<int64_t>(d.n_samples - 1, (int64_t)(rng.uniform() * (double)d.n_samples));
      arr.push_back(Arrival{t, d.kappa_bytes, (double)d.prompt_tokens[j], (double)d.output_tokens[j],
                            d.service_time_s[j]});
    }
  }
  std::stable_sort(arr.begin(), arr.end(), [](const Arrival &x, const Arrival &y) { return x.a < y.a; });

  std::vector<double> demand((size_t)opts->n_obs);
  for (int64_t k = 0; k < opts->n_obs; ++k) {
    const double t = W + rng.uniform() * (H - W);
    // arrivals in (t - W, t]: the only ones that can be active
    auto lo = std::upper_bound(arr.begin(), arr.end(), t - W, [](double v, const Arrival &x) { return v < x.a; });
    auto hi = std::upper_bound(lo, arr.end(), t, [](double v, const Arrival &x) { return v < x.a; });
    double sum = 0;
    for (auto it = lo; it != hi; ++it) {
      const double u = t - it->a;
      if (u >= 0 && u < it->tr) sum += it->kappa * (it->op + it->od * u / it->tr);
    }
    demand[(size_t)k] = sum;
  }
  double mean = 0, mx = 0;
  for (double v : demand) {
    mean += v;
    mx = std::max(mx, v);
  }
  mean /= (double)demand.size();
  std::sort(demand.begin(), demand.end());
  const int64_t rank = std::max<int64_t>(1, (int64_t)std::ceil(q * (double)demand.size()));
  const double qb = demand[(size_t)(rank - 1)];
  const double chunks = std::ceil(qb / (double)opts->chunk_bytes);
  if (chunks > 9.0e15 / (double)opts->chunk_bytes) return fail(CP_EINVAL, "planned pool too large");
  out->quantile_bytes = qb;
  out->mean_bytes = mean;
  out->max_bytes = mx;
  out->pool_bytes = (uint64_t)chunks * opts->chunk_bytes;
  out->n_arrivals = (int64_t)arr.size();
  return CP_OK;
}

}  // extern "C"
