// Host construction of the MSE-optimal Gaussian grid G_n^p (Sec. 3.2 and
// Alg. 2 of the paper: the grid is computed once per (n, p)). The paper uses
// the CLVQ procedure without giving its steps; this file runs Lloyd's
// algorithm, which minimises the same objective E||x - Q(x)||^2 over
// x ~ N(0, I_p), on a seeded sample.
//
// Must be compiled with -ffp-contract=off: distances are formed as
// (v0-g0)^2 + (v1-g1)^2 with separate roundings, the plain definition.

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <numeric>
#include <thread>
#include <vector>

#include "internal.h"

namespace higgs {
namespace {

// Standard normal p-vectors, row-major [num][p]: Box-Muller on consecutive
// 53-bit uniforms of the splitmix64 stream.
std::vector<double> gaussian_samples(uint64_t seed, int64_t num, int p) {
  const int64_t total = num * p;
  const int64_t pairs = (total + 1) / 2;
  std::vector<double> out(static_cast<size_t>(2 * pairs));
  const double twopi = 2.0 * M_PI;
  for (int64_t i = 0; i < pairs; ++i) {
    const double u1 = double(splitmix64_at(seed, uint64_t(2 * i)) >> 11) * 0x1p-53;
    const double u2 = double(splitmix64_at(seed, uint64_t(2 * i + 1)) >> 11) * 0x1p-53;
    const double r = std::sqrt(-2.0 * std::log(1.0 - u1));
    const double theta = twopi * u2;
    out[2 * i] = r * std::cos(theta);
    out[2 * i + 1] = r * std::sin(theta);
  }
  out.resize(static_cast<size_t>(total));
  return out;
}

// Exact nearest point with pruning: the points are visited outward from the
// sample's position in the list sorted by first coordinate, and a direction
// stops once (x0 - g0)^2 exceeds the best distance (no point further out can
// be closer). Ties keep the lowest index, as a full scan in index order does.
struct NearestSearch {
  int p = 0, n = 0;
  std::vector<double> key;      // first coordinate, sorted
  std::vector<int> order;       // grid index of each sorted entry
  const double* grid = nullptr;

  void build(const double* g, int p_, int n_) {
    grid = g;
    p = p_;
    n = n_;
    order.resize(n);
    std::iota(order.begin(), order.end(), 0);
    std::stable_sort(order.begin(), order.end(),
                     [&](int a, int b) { return g[a * p] < g[b * p]; });
    key.resize(n);
    for (int i = 0; i < n; ++i) key[i] = g[order[i] * p];
  }

  inline double dist(const double* v, int k) const {
    const double* gk = grid + k * p;
    double a = v[0] - gk[0];
    double d = a * a;
    for (int t = 1; t < p; ++t) {
      const double b = v[t] - gk[t];
      d = d + b * b;
    }
    return d;
  }

  inline void query(const double* v, int* best_k, double* best_d) const {
    int pos = int(std::lower_bound(key.begin(), key.end(), v[0]) - key.begin());
    int bk = -1;
    double bd = INFINITY;
    auto consider = [&](int s) -> bool {  // returns false when the direction can stop
      const double a = v[0] - key[s];
      if (a * a > bd) return false;
      const int k = order[s];
      const double d = dist(v, k);
      if (d < bd || (d == bd && k < bk)) {
        bd = d;
        bk = k;
      }
      return true;
    };
    int lo = pos - 1, hi = pos;
    bool go_lo = lo >= 0, go_hi = hi < n;
    while (go_lo || go_hi) {
      if (go_hi) {
        go_hi = consider(hi);
        ++hi;
        if (hi >= n) go_hi = false;
      }
      if (go_lo) {
        go_lo = consider(lo);
        --lo;
        if (lo < 0) go_lo = false;
      }
    }
    *best_k = bk;
    *best_d = bd;
  }
};

void assign_all(const NearestSearch& ns, const std::vector<double>& x, int64_t num, int p,
                std::vector<int>& assign, std::vector<double>& best) {
  unsigned hw = std::thread::hardware_concurrency();
  int threads = int(std::min<unsigned>(hw == 0 ? 1 : hw, 16));
  if (num < 65536) threads = 1;
  auto work = [&](int64_t a, int64_t b) {
    for (int64_t i = a; i < b; ++i) {
      int k;
      double d;
      ns.query(&x[size_t(i * p)], &k, &d);
      assign[size_t(i)] = k;
      best[size_t(i)] = d;
    }
  };
  if (threads == 1) {
    work(0, num);
    return;
  }
  std::vector<std::thread> pool;
  const int64_t step = (num + threads - 1) / threads;
  for (int t = 0; t < threads; ++t) {
    const int64_t a = t * step, b = std::min(num, a + step);
    if (a < b) pool.emplace_back(work, a, b);
  }
  for (auto& th : pool) th.join();
}

}  // namespace

int lloyd_grid(int p, int n, uint64_t seed, int64_t num_samples, int max_iters,
               double* grid_out, double* mse_out, int* iters_out) {
  const std::vector<double> x = gaussian_samples(seed, num_samples, p);
  std::vector<double> grid(x.begin(), x.begin() + size_t(n) * p);
  std::vector<int> assign(static_cast<size_t>(num_samples)), prev;
  std::vector<double> best(static_cast<size_t>(num_samples));
  std::vector<double> sums(static_cast<size_t>(n) * p);
  std::vector<int64_t> counts(static_cast<size_t>(n));
  NearestSearch ns;
  int iters = 0;
  for (;;) {
    ns.build(grid.data(), p, n);
    assign_all(ns, x, num_samples, p, assign, best);
    if (!prev.empty() && assign == prev) break;
    if (iters >= max_iters) break;
    // cell means, summed in sample order
    std::fill(sums.begin(), sums.end(), 0.0);
    std::fill(counts.begin(), counts.end(), 0);
    for (int64_t i = 0; i < num_samples; ++i) {
      const int k = assign[size_t(i)];
      counts[size_t(k)] += 1;
      for (int t = 0; t < p; ++t) sums[size_t(k) * p + t] += x[size_t(i * p + t)];
    }
    for (int k = 0; k < n; ++k) {
      if (counts[size_t(k)] == 0) continue;  // empty cell keeps its point
      for (int t = 0; t < p; ++t)
        grid[size_t(k) * p + t] = sums[size_t(k) * p + t] / double(counts[size_t(k)]);
    }
    prev.swap(assign);
    assign.resize(size_t(num_samples));
    ++iters;
  }
  double total = 0.0;
  for (int64_t i = 0; i < num_samples; ++i) total += best[size_t(i)];
  std::copy(grid.begin(), grid.end(), grid_out);
  if (mse_out) *mse_out = total / (double(num_samples) * p);
  if (iters_out) *iters_out = iters;
  return 0;
}


// ---------------------------------------------------------------------------
// Uniform grid (the CH8 format of Sec. 3.3: a grid constrained to be uniform,
// placed and scaled to minimise the expected squared error over N(0, 1)).
// Points c_k = step (k - (n - 1) / 2), k < n, symmetric about 0 (the optimum
// for a symmetric density); cell k is [t_k, t_{k+1}] with thresholds at the
// midpoints t_k = step (k - n / 2) and t_0 = -inf, t_n = +inf. With phi, Q the
// standard normal density and upper tail,
//   int_a^b (x - c)^2 phi = (1 + c^2) P(a, b) + a phi(a) - b phi(b)
//                           - 2 c (phi(a) - phi(b)),       P(a, b) = Q(a) - Q(b),
// and, the thresholds being midpoints, the boundary terms of dMSE/dstep cancel:
//   dMSE/dstep = -2 sum_k m_k [phi(t_k) - phi(t_{k+1}) - c_k P(t_k, t_{k+1})],
// m_k = k - (n - 1) / 2. The step is the root of that derivative (bisection
// to the last bit: the derivative changes sign once).
// ---------------------------------------------------------------------------
namespace {

double phi(double x) { return std::isinf(x) ? 0.0 : std::exp(-0.5 * x * x) / std::sqrt(2.0 * M_PI); }
double upper_tail(double x) { return 0.5 * std::erfc(x / std::sqrt(2.0)); }
// P(a, b) = Pr[a < X < b], formed from the tail on the side away from 0
double mass(double a, double b) {
  if (a >= 0.0) return upper_tail(a) - upper_tail(b);
  if (b <= 0.0) return upper_tail(-b) - upper_tail(-a);
  return 1.0 - upper_tail(-a) - upper_tail(b);
}

double uniform_mse(int n, double step) {
  double sum = 0.0;
  for (int k = 0; k < n; ++k) {
    const double c = step * (k - 0.5 * (n - 1));
    const double a = k == 0 ? -INFINITY : step * (k - 0.5 * n);
    const double b = k == n - 1 ? INFINITY : step * (k + 1 - 0.5 * n);
    const double aphi = std::isinf(a) ? 0.0 : a * phi(a);
    const double bphi = std::isinf(b) ? 0.0 : b * phi(b);
    sum += (1.0 + c * c) * mass(a, b) + aphi - bphi - 2.0 * c * (phi(a) - phi(b));
  }
  return sum;
}

double uniform_mse_slope(int n, double step) {
  double sum = 0.0;
  for (int k = 0; k < n; ++k) {
    const double m = k - 0.5 * (n - 1);
    const double c = step * m;
    const double a = k == 0 ? -INFINITY : step * (k - 0.5 * n);
    const double b = k == n - 1 ? INFINITY : step * (k + 1 - 0.5 * n);
    sum += m * (phi(a) - phi(b) - c * mass(a, b));
  }
  return -2.0 * sum;
}

}  // namespace

void uniform_grid(int n, double* grid_out, double* step_out, double* mse_out) {
  // the slope is negative for a tiny step (overload dominates) and positive
  // for a step past the support of N(0, 1)
  double lo = 1e-6, hi = 8.0;
  for (int it = 0; it < 200 && hi - lo > 0.0; ++it) {
    const double mid = 0.5 * (lo + hi);
    if (mid <= lo || mid >= hi) break;
    if (uniform_mse_slope(n, mid) < 0.0)
      lo = mid;
    else
      hi = mid;
  }
  const double step = 0.5 * (lo + hi);
  for (int k = 0; k < n; ++k) grid_out[k] = step * (k - 0.5 * (n - 1));
  if (step_out) *step_out = step;
  if (mse_out) *mse_out = uniform_mse(n, step);
}

}  // namespace higgs
