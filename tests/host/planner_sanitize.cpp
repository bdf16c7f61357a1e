// Host driver for the batch-planning calls, built with AddressSanitizer and
// UndefinedBehaviorSanitizer by tests/test_planner_sanitize.py: every call is
// exercised on seeded random batches and on the edge cases of its contract
// (empty, single, all-equal, out-of-range arguments), and the invariants of
// the results are checked.  A sanitizer report or a failed check exits non-zero.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <vector>

#include "darts.h"

namespace {

uint64_t g_state = 0x9e3779b97f4a7c15ull;
uint32_t next_u32() {
  g_state = g_state * 6364136223846793005ull + 1442695040888963407ull;
  return (uint32_t)(g_state >> 33);
}
double next_unit() { return (next_u32() + 0.5) / 4294967296.0; }

int g_fail = 0;
void check(bool ok, const char* what, int a = 0) {
  if (!ok) {
    std::fprintf(stderr, "check failed: %s (%d)\n", what, a);
    g_fail = 1;
  }
}

void allocation() {
  for (int trial = 0; trial < 200; ++trial) {
    const int n = 1 + (int)(next_u32() % 300);
    const int m_low = 1 + (int)(next_u32() % 8);
    const int m_up = m_low + (int)(next_u32() % 24);
    const int64_t m_total = (int64_t)n * m_low + (int64_t)(next_u32() % (uint32_t)(n * (m_up - m_low) + 5));
    std::vector<double> sigma(n);
    std::vector<uint8_t> seen(n);
    for (int i = 0; i < n; ++i) {
      sigma[i] = (trial % 7 == 0) ? 1.0 : next_unit() * 100.0;
      seen[i] = (next_u32() % 5) != 0;
    }
    std::vector<int32_t> plan(n, -1);
    const int st = darts_allocate_redundancy(sigma.data(), trial % 3 ? seen.data() : nullptr, n, m_low,
                                             m_up, m_total, plan.data());
    check(st == DARTS_OK, "allocate status", st);
    int64_t sum = 0;
    for (int i = 0; i < n; ++i) {
      check(plan[i] >= m_low && plan[i] <= m_up, "plan range", plan[i]);
      sum += plan[i];
    }
    const int64_t cap = (int64_t)n * m_up;
    check(sum == (m_total < cap ? m_total : cap), "plan sum", (int)sum);
  }
  // out-of-range arguments are rejected without writes
  std::vector<int32_t> plan(4, 7);
  double s4[4] = {1, 2, 3, 4};
  check(darts_allocate_redundancy(s4, nullptr, 4, 5, 4, 20, plan.data()) != DARTS_OK, "m_up < m_low");
  // a budget below n*m_low leaves every prompt at the floor m_low
  check(darts_allocate_redundancy(s4, nullptr, 4, 2, 4, 1, plan.data()) == DARTS_OK, "budget below n*m_low");
  for (int i = 0; i < 4; ++i) check(plan[i] == 2, "floor plan", plan[i]);
  check(darts_allocate_redundancy(nullptr, nullptr, 4, 2, 4, 12, plan.data()) != DARTS_OK, "null sigma");
}

void length_std_and_ema() {
  for (int trial = 0; trial < 100; ++trial) {
    const int n = 1 + (int)(next_u32() % 64), m = 1 + (int)(next_u32() % 32);
    std::vector<int32_t> len((size_t)n * m), plan(n);
    for (auto& l : len) l = (int32_t)(next_u32() % 20000);
    for (auto& p : plan) p = 1 + (int32_t)(next_u32() % (uint32_t)m);
    std::vector<double> sd(n, -1.0);
    check(darts_prompt_length_std(len.data(), trial % 2 ? plan.data() : nullptr, n, m, sd.data()) ==
              DARTS_OK, "length std status");
    for (int i = 0; i < n; ++i) check(sd[i] >= 0.0 && std::isfinite(sd[i]), "std finite", i);
    std::vector<double> est(n, 0.0), obs(n);
    std::vector<uint8_t> seen(n, 0);
    for (int i = 0; i < n; ++i) obs[i] = (i % 5 == 0) ? std::nan("") : sd[i];
    check(darts_ema_update(est.data(), seen.data(), obs.data(), n, 0.3) == DARTS_OK, "ema status");
    for (int i = 0; i < n; ++i) check(seen[i] == (i % 5 != 0), "ema seen", i);
  }
  double e = 0, o = 1;
  uint8_t s = 0;
  check(darts_ema_update(&e, &s, &o, 1, 0.0) != DARTS_OK, "alpha 0 rejected");
  check(darts_ema_update(&e, &s, &o, 1, 1.5) != DARTS_OK, "alpha > 1 rejected");
}

void budget() {
  for (int trial = 0; trial < 200; ++trial) {
    const int n = 1 + (int)(next_u32() % 512), M = 1 + (int)(next_u32() % 16);
    int64_t mt = -1;
    const double rho = next_unit() * 3.0, lam = (trial % 9 == 0) ? 0.0 : next_unit(),
                 kc = (trial % 11 == 0) ? 0.0 : next_unit() * 0.1;
    check(darts_redundancy_budget(rho, lam, kc, n, M, &mt) == DARTS_OK, "budget status");
    check(mt >= (int64_t)M * n && mt <= 2 * (int64_t)M * n, "budget clip", (int)mt);
  }
}

void cost_and_fit() {
  for (int trial = 0; trial < 40; ++trial) {
    const int n = (trial == 0) ? 0 : 1 + (int)(next_u32() % 2000);
    std::vector<int32_t> len(n), rank(n);
    for (int i = 0; i < n; ++i) {
      len[i] = (int32_t)(next_u32() % 10000);
      rank[i] = (int32_t)(next_u32() % 8);
    }
    const double ptl[6] = {64.0, 256.0, 5.0, 0.05, -0.01, -0.02};
    double T = -1.0, Tdp = -1.0;
    check(darts_rollout_cost(len.data(), n, ptl, &T) == DARTS_OK, "cost status");
    check(darts_rollout_cost_dp(len.data(), rank.data(), n, 8, ptl, &Tdp) == DARTS_OK, "cost dp status");
    check(T >= 0.0 && Tdp >= 0.0 && std::isfinite(T) && std::isfinite(Tdp), "cost finite");
    // a single rank is the plain Eq. 4
    std::vector<int32_t> zero(n, 0);
    double T1 = -1.0;
    check(darts_rollout_cost_dp(len.data(), zero.data(), n, 1, ptl, &T1) == DARTS_OK && T1 == T,
          "one rank equals Eq. 4");
    // steps of a random rollout, then the fit
    // (the fit is cubic in the distinct batch sizes: keep them to <= 48)
    const int steps = (trial % 5 == 0) ? 1 + trial % 4 : 50 + (int)(next_u32() % 400);
    std::vector<int32_t> bsz(steps);
    std::vector<double> lat(steps);
    for (int i = 0; i < steps; ++i) {
      bsz[i] = 1 + (int32_t)(next_u32() % 48) * 21;
      lat[i] = 4.0 + 0.04 * bsz[i] + next_unit();
    }
    double fit[6];
    check(darts_fit_ptl(bsz.data(), lat.data(), steps, fit) == DARTS_OK, "fit status");
    for (double v : fit) check(std::isfinite(v), "fit finite");
  }
  int32_t b = 3;
  double nan_lat = std::nan(""), fit[6];
  check(darts_fit_ptl(&b, &nan_lat, 1, fit) != DARTS_OK, "non-finite latency rejected");
  int32_t l2[2] = {3, 4}, r2[2] = {0, 9};
  const double ptl[6] = {1, 2, 1, 0, 0, 0};
  double T;
  check(darts_rollout_cost_dp(l2, r2, 2, 8, ptl, &T) != DARTS_OK, "rank out of range rejected");
}

}  // namespace

int main() {
  allocation();
  length_std_and_ema();
  budget();
  cost_and_fit();
  if (g_fail) return 1;
  std::printf("ok\n");
  return 0;
}
