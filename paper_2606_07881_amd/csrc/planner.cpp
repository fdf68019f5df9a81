// Host-only stage planning: the memory-constrained partition of a layer stack
// over pipeline stages (appendix "Memory-constrained pipeline partitioning")
// and the bubble-efficiency formulas of Eqs. (3)-(5).
#include <cmath>
#include <limits>
#include <vector>

#include "paci_stage.h"

namespace {

constexpr double kInf = std::numeric_limits<double>::infinity();

// Sums over the layers x .. i-1 for every 0 <= x < i <= L, accumulated left to
// right from layer x (so a sum is the same however it is looked up).
struct RangeSums {
  int L;
  std::vector<double> v;
  RangeSums(const double* f, int L_) : L(L_), v((size_t)(L_ + 1) * (L_ + 1), 0.0) {
    for (int x = 0; x < L; ++x) {
      double acc = 0.0;
      for (int i = x + 1; i <= L; ++i) {
        acc += f[i - 1];
        v[(size_t)x * (L + 1) + i] = acc;
      }
    }
  }
  double operator()(int x, int i) const { return v[(size_t)x * (L + 1) + i]; }
};

struct Problem {
  int L, N;
  double budget;
  RangeSums T, S, A;
  Problem(int L_, int N_, const double* t, const double* s, const double* a, double B)
      : L(L_), N(N_), budget(B), T(t, L_), S(s, L_), A(a, L_) {}
  // stage j (1-based) holding layers x .. i-1 keeps N - j + 1 micro-batches in flight
  double memory(int j, int x, int i) const { return S(x, i) + (double)(N - j + 1) * A(x, i); }
  double overshoot(int j, int x, int i) const { return std::max(0.0, memory(j, x, i) - budget); }
};

// Min-max dynamic program over prefixes: D[i][j] is the best value for the
// first i layers on the first j stages, a stage (x, i] costing cost(j, x, i),
// allowed only when its overshoot is at most `limit`. Fills cuts (N + 1
// entries) from the argmin table and returns the optimum (kInf if no prefix
// chain is allowed).
template <class Cost>
double minmax_dp(const Problem& p, double limit, Cost cost, int32_t* cuts) {
  const int L = p.L, N = p.N;
  std::vector<double> D((size_t)(L + 1) * (N + 1), kInf);
  std::vector<int> arg((size_t)(L + 1) * (N + 1), -1);
  auto at = [&](int i, int j) -> size_t { return (size_t)i * (N + 1) + j; };
  for (int i = 1; i <= L; ++i)
    if (p.overshoot(1, 0, i) <= limit) {
      D[at(i, 1)] = cost(1, 0, i);
      arg[at(i, 1)] = 0;
    }
  for (int j = 2; j <= N; ++j)
    for (int i = j; i <= L; ++i)
      for (int x = j - 1; x < i; ++x) {
        const double prev = D[at(x, j - 1)];
        if (prev == kInf || p.overshoot(j, x, i) > limit) continue;
        const double val = std::max(prev, cost(j, x, i));
        if (val < D[at(i, j)]) {
          D[at(i, j)] = val;
          arg[at(i, j)] = x;
        }
      }
  const double best = D[at(L, N)];
  if (best != kInf && cuts) {
    cuts[N] = L;
    for (int j = N, i = L; j >= 1; --j) {
      i = arg[at(i, j)];
      cuts[j - 1] = i;
    }
  }
  return best;
}

}  // namespace

extern "C" int paci_partition(int L, int N, const double* t, const double* s, const double* a, double budget,
                              int32_t* cuts, double* max_time, double* max_overshoot) {
  if (N < 1 || L < N || !t || !s || !a || !cuts || !(budget >= 0.0)) return PACI_E_INVAL;
  for (int l = 0; l < L; ++l)
    if (!(t[l] >= 0.0) || !(s[l] >= 0.0) || !(a[l] >= 0.0) || !std::isfinite(t[l]) || !std::isfinite(s[l]) ||
        !std::isfinite(a[l]))
      return PACI_E_INVAL;
  const Problem p(L, N, t, s, a, budget);
  auto time = [&](int, int x, int i) { return p.T(x, i); };
  auto over = [&](int j, int x, int i) { return p.overshoot(j, x, i); };
  // first pass: every stage within the budget
  double best = minmax_dp(p, 0.0, time, cuts);
  double worst_over = 0.0;
  if (best == kInf) {
    // fallback: the least largest overshoot, then the least largest stage time
    // among the partitions that reach it
    worst_over = minmax_dp(p, kInf, over, nullptr);
    best = minmax_dp(p, worst_over, time, cuts);
  }
  if (max_time) *max_time = best;
  if (max_overshoot) *max_overshoot = worst_over;
  return PACI_OK;
}

extern "C" double paci_eta_flush(double m, int N) {
  if (!(m > 0.0) || N < 1) return std::nan("");
  return m / (m + (N - 1));
}

extern "C" double paci_eta_interleaved(double m, int N, int V) {
  if (!(m > 0.0) || N < 1 || V < 1) return std::nan("");
  return m * V / (m * V + (N - 1));
}

extern "C" double paci_throughput_proxy(double t_flush, double m, int N) {
  return t_flush / paci_eta_flush(m, N);
}
