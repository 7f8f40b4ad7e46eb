// Per-layer choice of quantizers under an average-bits budget (Sec. 4,
// "Variable Bitwidth Quantization", Eq. (objective)):
//   minimise  sum_l alpha_l * t2[l][j_l]
//   subject to sum_l bits[j_l] * d_l <= b_max * sum_l d_l.
// The paper solves it with an ILP solver; here it is solved exactly as a
// multiple-choice knapsack by dynamic programming over integer costs.
// Every HIGGS option costs log2(n)/p + 16/g bits per weight with g >= 64, a
// multiple of 2^-8, so cost[l][j] = bits[j] * 256 * d_l is an integer; all
// costs and the budget are divided by their greatest common divisor, and the
// table runs over the budget left above every layer's cheapest option
// ("slack"), capped where every layer can take its lowest-error option.
// Ties keep the lower option index (strict comparison), so the result is
// deterministic.

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <limits>
#include <numeric>
#include <vector>

#include "internal.h"

namespace higgs {

namespace {
constexpr int64_t kMaxTableBytes = int64_t(512) << 20;  // choice table limit
}

namespace {

int allocate_bits_impl(int layers, int options, const double* alpha, const double* t2,
                       const double* bits, const int64_t* sizes, double b_max, int32_t* choice,
                       double* objective, double* avg_bits, char* msg, int msg_len) {
  const int L = layers, J = options;
  if (L < 1 || J < 1 || J > 255) {
    std::snprintf(msg, size_t(msg_len), "need layers >= 1 and 1 <= options <= 255");
    return HIGGS_ERR_INVALID_ARG;
  }
  // integer cost units: bits * 256 per weight
  std::vector<int64_t> k(static_cast<size_t>(J));
  for (int j = 0; j < J; ++j) {
    const double v = bits[j] * 256.0;
    if (!(bits[j] > 0.0) || std::fabs(v - std::nearbyint(v)) > 1e-9 || v > double(1 << 20)) {
      std::snprintf(msg, size_t(msg_len),
                    "bits[%d]=%.17g must be a positive multiple of 2^-8 below 4096", j, bits[j]);
      return HIGGS_ERR_INVALID_ARG;
    }
    k[size_t(j)] = int64_t(std::nearbyint(v));
  }
  int64_t total = 0;
  for (int l = 0; l < L; ++l) {
    if (sizes[l] < 1 || sizes[l] > (int64_t(1) << 40)) {
      std::snprintf(msg, size_t(msg_len), "sizes[%d] must be in [1, 2^40]", l);
      return HIGGS_ERR_INVALID_ARG;
    }
    total += sizes[l];
    if (total > (int64_t(1) << 42)) {
      std::snprintf(msg, size_t(msg_len), "total size above 2^42 weights");
      return HIGGS_ERR_INVALID_ARG;
    }
  }
  // costs and budget, exact integers
  std::vector<int64_t> cost(size_t(L) * size_t(J));
  int64_t u = 0;
  for (int l = 0; l < L; ++l)
    for (int j = 0; j < J; ++j) {
      const int64_t c = k[size_t(j)] * sizes[l];
      cost[size_t(l) * J + j] = c;
      u = std::gcd(u, c);
    }
  const long double budget_ld = std::floor((long double)(b_max) * 256.0L * (long double)(total));
  if (!(budget_ld >= 0.0L)) {
    std::snprintf(msg, size_t(msg_len), "b_max must be >= 0");
    return HIGGS_ERR_INVALID_ARG;
  }
  const long double cap_ld = (long double)(std::numeric_limits<int64_t>::max() / 4);
  const int64_t budget = int64_t(std::min(budget_ld, cap_ld)) / u;
  for (auto& c : cost) c /= u;

  // slack above the cheapest options; enough slack for every best option
  int64_t base = 0, need = 0;
  std::vector<int64_t> mincost(static_cast<size_t>(L));
  for (int l = 0; l < L; ++l) {
    int64_t mn = cost[size_t(l) * J], best_c = cost[size_t(l) * J];
    double best_e = alpha[l] * t2[size_t(l) * J];
    for (int j = 1; j < J; ++j) {
      const int64_t c = cost[size_t(l) * J + j];
      mn = std::min(mn, c);
      const double e = alpha[l] * t2[size_t(l) * J + j];
      if (e < best_e) {
        best_e = e;
        best_c = c;
      }
    }
    mincost[size_t(l)] = mn;
    base += mn;
    need += best_c - mn;
  }
  if (budget < base) {
    std::snprintf(msg, size_t(msg_len),
                  "b_max=%.6g is below the cheapest assignment (%.6g bits per weight)", b_max,
                  double(base) * double(u) / 256.0 / double(total));
    return HIGGS_ERR_INVALID_ARG;
  }
  const int64_t cap = std::min(budget - base, need);
  // (cap + 1) * L entries, compared without forming the product (cap can
  // reach 2^62 when the sizes share no common divisor)
  if (cap >= kMaxTableBytes / int64_t(L)) {
    std::snprintf(msg, size_t(msg_len),
                  "budget table of %lld x %d entries exceeds the %lld MiB limit",
                  (long long)(cap + 1), L, (long long)(kMaxTableBytes >> 20));
    return HIGGS_ERR_UNSUPPORTED;
  }

  // f[c]: least objective of the layers so far with extra cost <= c
  std::vector<double> f(size_t(cap + 1), 0.0), g(size_t(cap + 1));
  std::vector<uint8_t> pick(size_t(cap + 1) * size_t(L));
  const double inf = std::numeric_limits<double>::infinity();
  for (int l = 0; l < L; ++l) {
    uint8_t* pl = pick.data() + size_t(l) * size_t(cap + 1);
    for (int64_t c = 0; c <= cap; ++c) {
      double best = inf;
      int bj = 0;
      for (int j = 0; j < J; ++j) {
        const int64_t e = cost[size_t(l) * J + j] - mincost[size_t(l)];
        if (e > c) continue;
        const double v = f[size_t(c - e)] + alpha[l] * t2[size_t(l) * J + j];
        if (v < best) {
          best = v;
          bj = j;
        }
      }
      g[size_t(c)] = best;
      pl[c] = uint8_t(bj);
    }
    f.swap(g);
  }
  // trace back from the full slack
  int64_t c = cap;
  double obj = 0.0, used = 0.0;
  for (int l = L - 1; l >= 0; --l) {
    const int j = pick[size_t(l) * size_t(cap + 1) + size_t(c)];
    choice[l] = j;
    c -= cost[size_t(l) * J + j] - mincost[size_t(l)];
  }
  for (int l = 0; l < L; ++l) {
    obj += alpha[l] * t2[size_t(l) * J + choice[l]];
    used += bits[choice[l]] * double(sizes[l]);
  }
  if (objective) *objective = obj;
  if (avg_bits) *avg_bits = used / double(total);
  return HIGGS_OK;
}

}  // namespace

// Every host allocation above is a std::vector: a failure throws, and no
// exception may leave the library.
int allocate_bits(int layers, int options, const double* alpha, const double* t2,
                  const double* bits, const int64_t* sizes, double b_max, int32_t* choice,
                  double* objective, double* avg_bits, char* msg, int msg_len) {
  try {
    return allocate_bits_impl(layers, options, alpha, t2, bits, sizes, b_max, choice, objective,
                              avg_bits, msg, msg_len);
  } catch (...) {
    std::snprintf(msg, size_t(msg_len), "host allocation failed");
    return HIGGS_ERR_DEVICE;
  }
}

}  // namespace higgs
