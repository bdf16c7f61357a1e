// Host-side planning that runs once per rollout batch, before the decode loop:
// adaptive redundancy allocation (paper Sec. 4.2.2, App. C / Alg. 1), the
// adaptive total budget (App. B), the smoothed per-prompt length spread it
// feeds on, and the rollout cost model (Sec. 4.2.1, Eq. 4) with its per-token
// latency curve fitted from measured decode steps (App. A).
//
// Plain C++ on purpose: these are O(N log N) decisions over a batch of
// prompts (or a few hundred measured steps), far off the GPU's critical path.
// All arithmetic is float64 with no contraction, so results are reproducible
// bit for bit.
#pragma STDC FP_CONTRACT OFF

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <queue>
#include <vector>

#include "../../include/darts.h"

namespace {

// Marginal decrease of the objective sum_i w_i / M'_i when M'_i grows by one.
inline double marginal_gain(double w, int m) { return w * (1.0 / m - 1.0 / (m + 1)); }

struct Cand {
  double gain;
  int32_t idx;
};
// max-heap order: larger gain first, then the lower prompt index
struct CandLess {
  bool operator()(const Cand& a, const Cand& b) const {
    if (a.gain != b.gain) return a.gain < b.gain;
    return a.idx > b.idx;
  }
};

}  // namespace

extern "C" {

int darts_prompt_length_std(const int32_t* h_len, const int32_t* h_plan, int32_t n_prompts,
                            int32_t m, double* h_std) {
  if (!h_len || !h_std || n_prompts < 0 || m < 1) return DARTS_EINVAL;
  for (int32_t i = 0; i < n_prompts; ++i) {
    const int32_t mi = h_plan ? h_plan[i] : m;
    if (mi < 0 || mi > m) return DARTS_EINVAL;
    double s = 0.0;
    for (int32_t j = 0; j < mi; ++j) s += (double)h_len[(int64_t)i * m + j];
    const double mu = mi > 0 ? s / mi : 0.0;
    double v = 0.0;
    for (int32_t j = 0; j < mi; ++j) {
      const double d = (double)h_len[(int64_t)i * m + j] - mu;
      v += d * d;
    }
    h_std[i] = mi > 0 ? std::sqrt(v / mi) : 0.0;
  }
  return DARTS_OK;
}

int darts_ema_update(double* h_est, uint8_t* h_seen, const double* h_obs, int32_t n, double alpha) {
  if (!h_est || !h_seen || !h_obs || n < 0 || !(alpha > 0.0 && alpha <= 1.0)) return DARTS_EINVAL;
  for (int32_t i = 0; i < n; ++i) {
    const double o = h_obs[i];
    if (std::isnan(o)) continue;
    h_est[i] = h_seen[i] ? alpha * o + (1.0 - alpha) * h_est[i] : o;
    h_seen[i] = 1;
  }
  return DARTS_OK;
}

int darts_redundancy_budget(double rho, double lambda, double k_cost, int32_t n_prompts, int32_t M,
                            int64_t* h_m_total) {
  if (!h_m_total || n_prompts < 0 || M < 1 || std::isnan(rho)) return DARTS_EINVAL;
  const int64_t lo = (int64_t)M * n_prompts, hi = 2 * lo;
  if (!(lambda > 0.0 && k_cost > 0.0)) { *h_m_total = hi; return DARTS_OK; }
  const double star = rho / (lambda * k_cost);
  if (!std::isfinite(star)) { *h_m_total = star > 0 ? hi : lo; return DARTS_OK; }
  const double f = std::floor(star);
  *h_m_total = f <= (double)lo ? lo : (f >= (double)hi ? hi : (int64_t)f);
  return DARTS_OK;
}

int darts_allocate_redundancy(const double* h_sigma, const uint8_t* h_seen, int32_t n_prompts,
                              int32_t m_low, int32_t m_up, int64_t m_total, int32_t* h_plan) {
  if (!h_sigma || !h_plan || n_prompts < 0 || m_low < 1 || m_up < m_low) return DARTS_EINVAL;
  if (n_prompts == 0) return DARTS_OK;
  // prompts never observed take the mean spread of the observed ones
  std::vector<double> s(h_sigma, h_sigma + n_prompts);
  if (h_seen) {
    double sum = 0.0;
    int cnt = 0;
    for (int32_t i = 0; i < n_prompts; ++i)
      if (h_seen[i]) { sum += s[i]; ++cnt; }
    const double mean = cnt > 0 ? sum / cnt : 0.0;
    for (int32_t i = 0; i < n_prompts; ++i)
      if (!h_seen[i]) s[i] = mean;
  }
  for (double v : s)
    if (!std::isfinite(v)) return DARTS_EINVAL;
  // Alg. 1 line 1: min-max normalised weights (all equal -> 1)
  const double lo = *std::min_element(s.begin(), s.end());
  const double hi = *std::max_element(s.begin(), s.end());
  std::vector<double> w(n_prompts);
  for (int32_t i = 0; i < n_prompts; ++i) w[i] = hi == lo ? 1.0 : (s[i] - lo) / (hi - lo);
  // lines 1-2: every prompt starts at M_low; lines 3-7: hand out the rest one
  // unit at a time to the largest marginal gain (ties: lowest index).  A heap
  // over prompts below M_up yields the same sequence of choices as a scan.
  std::priority_queue<Cand, std::vector<Cand>, CandLess> heap;
  for (int32_t i = 0; i < n_prompts; ++i) {
    h_plan[i] = m_low;
    if (m_low < m_up) heap.push({marginal_gain(w[i], m_low), i});
  }
  int64_t remain = m_total - (int64_t)n_prompts * m_low;
  while (remain > 0 && !heap.empty()) {
    const Cand c = heap.top();
    heap.pop();
    const int32_t i = c.idx;
    h_plan[i] += 1;
    --remain;
    if (h_plan[i] < m_up) heap.push({marginal_gain(w[i], h_plan[i]), i});
  }
  return DARTS_OK;
}

}  // extern "C"
