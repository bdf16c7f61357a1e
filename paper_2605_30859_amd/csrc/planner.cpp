// Host-side planning that runs once per rollout batch, before the decode loop:
// adaptive redundancy allocation (paper Sec. 4.2.2, App. C / Alg. 1), the
// adaptive total budget (App. B), the smoothed per-prompt length spread it
// feeds on, and the rollout cost model (Sec. 4.2.1, Eq. 4) with its per-token
// latency curve fitted from measured decode steps (App. A).
//
// Plain C++ on purpose: these are O(N log N) decisions over a batch of
// prompts or cubic in the distinct batch sizes of a few thousand measured
// steps, far off the GPU's critical path.
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

// ---------------------------------------------------------------- cost model
// PTL(b) = c0 + c1 b + c2 max(0, b - b1) + c3 max(0, b - b2); p = {b1, b2, c0, c1, c2, c3}
static inline double ptl_eval(const double* p, double b) {
  return p[2] + p[3] * b + p[4] * std::max(0.0, b - p[0]) + p[5] * std::max(0.0, b - p[1]);
}

int darts_rollout_cost(const int32_t* h_len, int32_t n, const double* h_ptl, double* h_T) {
  if ((!h_len && n > 0) || !h_ptl || !h_T || n < 0) return DARTS_EINVAL;
  std::vector<int32_t> l(h_len, h_len + n);
  std::sort(l.begin(), l.end());
  // Eq. 4: between consecutive completions, (l_[m] - l_[m-1]) steps at batch n - m + 1
  double T = 0.0;
  int32_t prev = 0;
  for (int32_t m = 1; m <= n; ++m) {
    T += (double)(l[m - 1] - prev) * ptl_eval(h_ptl, (double)(n - m + 1));
    prev = l[m - 1];
  }
  *h_T = T;
  return DARTS_OK;
}

int darts_rollout_cost_dp(const int32_t* h_len, const int32_t* h_rank, int32_t n, int32_t n_ranks,
                          const double* h_ptl, double* h_T) {
  if (n < 0 || n_ranks < 1 || ((!h_len || !h_rank) && n > 0) || !h_ptl || !h_T) return DARTS_EINVAL;
  std::vector<std::vector<int32_t>> per(n_ranks);
  for (int32_t i = 0; i < n; ++i) {
    if (h_rank[i] < 0 || h_rank[i] >= n_ranks) return DARTS_EINVAL;
    per[h_rank[i]].push_back(h_len[i]);
  }
  // the slowest rank sets the batch cost (an empty rank costs 0)
  double T = 0.0;
  for (int32_t r = 0; r < n_ranks; ++r) {
    double t = 0.0;
    const int rc = darts_rollout_cost(per[r].data(), (int32_t)per[r].size(), h_ptl, &t);
    if (rc != DARTS_OK) return rc;
    T = r == 0 ? t : std::max(T, t);
  }
  *h_T = T;
  return DARTS_OK;
}

namespace {
// Weighted least squares of the hinge basis (1, x, (x-b1)+, (x-b2)+) on the
// per-size mean latencies (weights = sample counts; the same solution as the
// raw samples).  x is scaled by 1/s for conditioning.  Returns false if the
// 4x4 normal system is singular.
bool hinge_lsq(const std::vector<double>& xs, const std::vector<double>& cnt,
               const std::vector<double>& mean, double b1, double b2, double s, double c[4]) {
  double A[4][5] = {};
  for (size_t k = 0; k < xs.size(); ++k) {
    const double x = xs[k] / s;
    const double f[4] = {1.0, x, std::max(0.0, x - b1 / s), std::max(0.0, x - b2 / s)};
    for (int r = 0; r < 4; ++r) {
      for (int q = 0; q < 4; ++q) A[r][q] += cnt[k] * f[r] * f[q];
      A[r][4] += cnt[k] * f[r] * mean[k];
    }
  }
  for (int col = 0; col < 4; ++col) {          // Gaussian elimination, partial pivoting
    int piv = col;
    for (int r = col + 1; r < 4; ++r)
      if (std::fabs(A[r][col]) > std::fabs(A[piv][col])) piv = r;
    if (A[piv][col] == 0.0) return false;
    if (piv != col)
      for (int q = 0; q < 5; ++q) std::swap(A[col][q], A[piv][q]);
    for (int r = col + 1; r < 4; ++r) {
      const double f = A[r][col] / A[col][col];
      for (int q = col; q < 5; ++q) A[r][q] -= f * A[col][q];
    }
  }
  for (int r = 3; r >= 0; --r) {
    double v = A[r][4];
    for (int q = r + 1; q < 4; ++q) v -= A[r][q] * c[q];
    c[r] = v / A[r][r];
  }
  // back to unscaled batch sizes
  c[1] /= s; c[2] /= s; c[3] /= s;
  return true;
}
}  // namespace

int darts_fit_ptl(const int32_t* h_bsz, const double* h_lat, int32_t n, double* h_ptl) {
  if ((n > 0 && (!h_bsz || !h_lat)) || !h_ptl || n < 0) return DARTS_EINVAL;
  // distinct sizes with sample counts and mean latency
  std::vector<std::pair<int32_t, double>> v(n);
  for (int32_t i = 0; i < n; ++i) {
    if (!std::isfinite(h_lat[i])) return DARTS_EINVAL;
    v[i] = {h_bsz[i], h_lat[i]};
  }
  std::sort(v.begin(), v.end(), [](const auto& a, const auto& b) { return a.first < b.first; });
  std::vector<double> xs, cnt, mean;
  for (int32_t i = 0; i < n;) {
    int32_t j = i;
    double sum = 0.0;
    while (j < n && v[j].first == v[i].first) sum += v[j++].second;
    xs.push_back((double)v[i].first);
    cnt.push_back((double)(j - i));
    mean.push_back(sum / (j - i));
    i = j;
  }
  const int D = (int)xs.size();
  for (int q = 0; q < 6; ++q) h_ptl[q] = 0.0;
  if (D == 0) return DARTS_OK;
  if (D == 1) { h_ptl[0] = h_ptl[1] = xs[0]; h_ptl[2] = mean[0]; return DARTS_OK; }
  if (D < 4) {
    // one weighted least-squares line
    double sw = 0, sx = 0, sy = 0, sxx = 0, sxy = 0;
    for (int k = 0; k < D; ++k) {
      sw += cnt[k]; sx += cnt[k] * xs[k]; sy += cnt[k] * mean[k];
      sxx += cnt[k] * xs[k] * xs[k]; sxy += cnt[k] * xs[k] * mean[k];
    }
    const double den = sw * sxx - sx * sx;
    h_ptl[0] = h_ptl[1] = xs[D - 1];
    h_ptl[3] = (sw * sxy - sx * sy) / den;
    h_ptl[2] = (sy - h_ptl[3] * sx) / sw;
    return DARTS_OK;
  }
  const double s = xs[D - 1] > 0 ? xs[D - 1] : 1.0;
  double best = INFINITY;
  for (int i = 1; i <= D - 3; ++i)
    for (int j = i + 1; j <= D - 2; ++j) {
      double c[4];
      if (!hinge_lsq(xs, cnt, mean, xs[i], xs[j], s, c)) continue;
      const double p[6] = {xs[i], xs[j], c[0], c[1], c[2], c[3]};
      double sse = 0.0;                        // between-size part of the residual
      for (int k = 0; k < D; ++k) {
        const double r = mean[k] - ptl_eval(p, xs[k]);
        sse += cnt[k] * r * r;
      }
      if (sse < best) {
        best = sse;
        for (int q = 0; q < 6; ++q) h_ptl[q] = p[q];
      }
    }
  return DARTS_OK;
}

}  // extern "C"
