// Redline selection (paper §4.2 steps (ii)-(iv), App. A): violation counts,
// exact binomial p-values, Holm step-down, fastest valid configuration.
// Host-only C++; no device work.
#include <math.h>
#include <stdint.h>

#include <algorithm>
#include <numeric>
#include <string>
#include <vector>

#include "../../include/bd.h"

namespace bd {
void set_error(const char* msg);   // defined with bd_last_error
}

namespace {

// Pr[Bin(n, a) <= v] summed term by term in long double.  Each term is
// exp(log C(n, j) + j log a + (n - j) log(1 - a)) and the sum is formed
// relative to the largest term, so no term under- or overflows before the
// final scaling; the relative error stays below 1e-13 for n <= 1e6.
long double binom_cdf(int64_t n, double alpha, int64_t v) {
  if (v < 0) return 0.0L;
  if (v >= n) return 1.0L;
  const long double la = logl((long double)alpha), lb = log1pl(-(long double)alpha);
  const long double lgn = lgammal((long double)n + 1.0L);
  std::vector<long double> lt((size_t)v + 1);
  long double mx = -INFINITY;
  for (int64_t j = 0; j <= v; ++j) {
    lt[(size_t)j] = lgn - lgammal((long double)j + 1.0L) - lgammal((long double)(n - j) + 1.0L) +
                    (long double)j * la + (long double)(n - j) * lb;
    mx = std::max(mx, lt[(size_t)j]);
  }
  long double s = 0.0L;
  for (int64_t j = 0; j <= v; ++j) s += expl(lt[(size_t)j] - mx);
  long double p = expl(mx) * s;
  return p > 1.0L ? 1.0L : p;
}

}  // namespace

extern "C" bd_status rl_risk_select(int32_t n, int32_t m, int32_t ref_index, const uint8_t* correct,
                                    const double* cost, double alpha, double delta, int32_t* V_out,
                                    double* p_out, uint8_t* valid_out, int32_t* selected_out,
                                    int32_t* near_ties_out) {
  if (n < 1 || m < 1 || ref_index < 0 || ref_index >= m || !correct || !cost || !selected_out) {
    bd::set_error("rl_risk_select: need n, m >= 1, ref_index in [0, m) and non-NULL inputs");
    return BD_EINVAL;
  }
  if (!(alpha > 0.0 && alpha < 1.0) || !(delta > 0.0 && delta <= 1.0)) {
    bd::set_error("rl_risk_select: need 0 < alpha < 1 and 0 < delta <= 1");
    return BD_EINVAL;
  }
  std::vector<int64_t> V(m, 0);
  const uint8_t* ref = correct + (size_t)ref_index * n;
  for (int j = 0; j < m; ++j) {
    const uint8_t* c = correct + (size_t)j * n;
    int64_t k = 0;
    for (int i = 0; i < n; ++i) k += (ref[i] != 0) && (c[i] == 0);
    V[j] = k;
  }
  std::vector<long double> p(m);
  for (int j = 0; j < m; ++j) p[j] = binom_cdf(n, alpha, V[j]);
  // Holm: ascending p, index order among equals; reject while p_(i) <= delta / (m - i + 1).
  std::vector<int> order(m);
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return p[a] < p[b]; });
  std::vector<uint8_t> valid(m, 0);
  int near = 0;
  for (int i = 0; i < m; ++i) {
    const int j = order[i];
    const long double thr = (long double)delta / (long double)(m - i);
    if (fabsl(p[j] / thr - 1.0L) < 1e-9L) ++near;
    if (p[j] <= thr) valid[j] = 1;
    else break;
  }
  int best = -1;
  for (int j = 0; j < m; ++j)
    if (valid[j] && (best < 0 || cost[j] > cost[best])) best = j;
  *selected_out = best < 0 ? ref_index : best;
  for (int j = 0; j < m; ++j) {
    if (V_out) V_out[j] = (int32_t)V[j];
    if (p_out) p_out[j] = (double)p[j];
    if (valid_out) valid_out[j] = valid[j];
  }
  if (near_ties_out) *near_ties_out = near;
  return BD_OK;
}
