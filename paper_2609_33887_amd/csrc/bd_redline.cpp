// Redline selection (paper §4.2 steps (ii)-(iv), App. A): violation counts,
// exact binomial p-values, Holm step-down, fastest valid configuration; the
// other procedures of App. A.3 and the baselines of App. D, the budget sweep
// (App. A.6), split-half exceedance (§5, App. D) and the Monte Carlo check
// with known risks (App. A.7).  Host-only C++ (splits and trials run on host
// threads); no device work.
#include <math.h>
#include <stdint.h>

#include <stdio.h>

#include <algorithm>
#include <numeric>
#include <string>
#include <thread>
#include <unordered_map>
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

// Procedures of App. A.3 and the baselines of App. D on p-values p (and
// counts V over n prompts for the plug-in rule).  valid gets 0/1; near (Holm
// only) counts comparisons whose ratio p / threshold is within 1e-9 of 1.
void valid_set(int method, int m, const long double* p, const int64_t* V, int64_t n, double alpha,
               double delta, const int32_t* order, uint8_t* valid, int* near) {
  std::fill(valid, valid + m, 0);
  if (near) *near = 0;
  switch (method) {
    case RL_HOLM: {
      // ascending p, index order among equals; reject while p_(i) <= delta / (m - i + 1)
      std::vector<int> ord(m);
      std::iota(ord.begin(), ord.end(), 0);
      std::stable_sort(ord.begin(), ord.end(), [&](int a, int b) { return p[a] < p[b]; });
      for (int i = 0; i < m; ++i) {
        const int j = ord[i];
        const long double thr = (long double)delta / (long double)(m - i);
        if (near && fabsl(p[j] / thr - 1.0L) < 1e-9L) ++*near;
        if (p[j] <= thr) valid[j] = 1;
        else break;
      }
      break;
    }
    case RL_BONFERRONI:
      for (int j = 0; j < m; ++j) valid[j] = p[j] <= (long double)delta / (long double)m;
      break;
    case RL_FIXED_SEQUENCE:
      for (int i = 0; i < m; ++i) {
        if (p[order[i]] <= (long double)delta) valid[order[i]] = 1;
        else break;
      }
      break;
    case RL_UNCORRECTED:
      for (int j = 0; j < m; ++j) valid[j] = p[j] <= (long double)delta;
      break;
    default:  // RL_PLUGIN
      for (int j = 0; j < m; ++j) valid[j] = (double)V[j] / (double)n <= alpha;
  }
}

// fastest valid configuration, lowest index among equals; the reference if none
int deploy(int m, const double* cost, const uint8_t* valid, int ref) {
  int best = -1;
  for (int j = 0; j < m; ++j)
    if (valid[j] && (best < 0 || cost[j] > cost[best])) best = j;
  return best < 0 ? ref : best;
}

// p-values Pr[Bin(n, alpha) <= v], memoised per (n, v) for one alpha
struct PvalCache {
  double alpha;
  std::unordered_map<int64_t, long double> memo;
  explicit PvalCache(double a) : alpha(a) {}
  long double operator()(int64_t n, int64_t v) {
    const int64_t key = n * (int64_t)2147483648LL + v;
    auto it = memo.find(key);
    if (it != memo.end()) return it->second;
    const long double p = binom_cdf(n, alpha, v);
    memo.emplace(key, p);
    return p;
  }
};

// violation bits ref & !c_j, packed 64 prompts per word
struct ViolBits {
  int m, n, words;
  std::vector<uint64_t> bits;   // [m][words]
  ViolBits(int m_, int n_, int ref, const uint8_t* correct) : m(m_), n(n_), words((n_ + 63) / 64) {
    bits.assign((size_t)m * words, 0);
    const uint8_t* r = correct + (size_t)ref * n;
    for (int j = 0; j < m; ++j) {
      const uint8_t* c = correct + (size_t)j * n;
      uint64_t* w = &bits[(size_t)j * words];
      for (int i = 0; i < n; ++i)
        if (r[i] != 0 && c[i] == 0) w[i >> 6] |= 1ull << (i & 63);
    }
  }
  // violations of configuration j on the prompts of mask (all when NULL)
  int64_t count(int j, const uint64_t* mask) const {
    const uint64_t* w = &bits[(size_t)j * words];
    int64_t k = 0;
    for (int q = 0; q < words; ++q) k += __builtin_popcountll(mask ? (w[q] & mask[q]) : w[q]);
    return k;
  }
};

std::vector<uint64_t> pack_mask(const uint8_t* mask, int n, bool invert) {
  std::vector<uint64_t> w((n + 63) / 64, 0);
  for (int i = 0; i < n; ++i)
    if ((mask[i] != 0) != invert) w[i >> 6] |= 1ull << (i & 63);
  return w;
}

bool check_common(const char* fn, int32_t n, int32_t m, int32_t ref_index, const void* correct,
                  const double* cost, double alpha, double delta, int32_t method, const int32_t* order) {
  char msg[256];
  if (n < 1 || m < 1 || ref_index < 0 || ref_index >= m || !correct || !cost) {
    snprintf(msg, sizeof msg, "%s: need n, m >= 1, ref_index in [0, m) and non-NULL inputs", fn);
    bd::set_error(msg);
    return false;
  }
  if (!(alpha > 0.0 && alpha < 1.0) || !(delta > 0.0 && delta <= 1.0)) {
    snprintf(msg, sizeof msg, "%s: need 0 < alpha < 1 and 0 < delta <= 1", fn);
    bd::set_error(msg);
    return false;
  }
  if (method < RL_HOLM || method > RL_PLUGIN) {
    snprintf(msg, sizeof msg, "%s: unknown procedure %d", fn, method);
    bd::set_error(msg);
    return false;
  }
  if (method == RL_FIXED_SEQUENCE) {
    std::vector<uint8_t> seen(m, 0);
    bool ok = order != nullptr;
    for (int i = 0; ok && i < m; ++i) {
      ok = order[i] >= 0 && order[i] < m && !seen[order[i]];
      if (ok) seen[order[i]] = 1;
    }
    if (!ok) {
      snprintf(msg, sizeof msg, "%s: the fixed sequence needs an order that is a permutation of 0..m-1", fn);
      bd::set_error(msg);
      return false;
    }
  }
  return true;
}

// run fn(i) for i in [0, count) on up to hardware_concurrency threads
template <class F>
void parallel_for(int count, F fn) {
  int nt = (int)std::min<unsigned>(std::max(1u, std::thread::hardware_concurrency()), 64u);
  nt = std::min(nt, std::max(1, count / 8));
  if (nt <= 1) {
    for (int i = 0; i < count; ++i) fn(i, 0);
    return;
  }
  std::vector<std::thread> th;
  for (int t = 0; t < nt; ++t)
    th.emplace_back([&, t] {
      for (int i = t; i < count; i += nt) fn(i, t);
    });
  for (auto& x : th) x.join();
}

}  // namespace

extern "C" bd_status rl_risk_select(int32_t n, int32_t m, int32_t ref_index, const uint8_t* correct,
                                    const double* cost, double alpha, double delta, int32_t* V_out,
                                    double* p_out, uint8_t* valid_out, int32_t* selected_out,
                                    int32_t* near_ties_out) {
  if (!check_common("rl_risk_select", n, m, ref_index, correct, cost, alpha, delta, RL_HOLM, nullptr) ||
      !selected_out) {
    if (!selected_out) bd::set_error("rl_risk_select: selected_out is NULL");
    return BD_EINVAL;
  }
  ViolBits vb(m, n, ref_index, correct);
  std::vector<int64_t> V(m);
  std::vector<long double> p(m);
  for (int j = 0; j < m; ++j) {
    V[j] = vb.count(j, nullptr);
    p[j] = binom_cdf(n, alpha, V[j]);
  }
  std::vector<uint8_t> valid(m);
  int near = 0;
  valid_set(RL_HOLM, m, p.data(), V.data(), n, alpha, delta, nullptr, valid.data(), &near);
  *selected_out = deploy(m, cost, valid.data(), ref_index);
  for (int j = 0; j < m; ++j) {
    if (V_out) V_out[j] = (int32_t)V[j];
    if (p_out) p_out[j] = (double)p[j];
    if (valid_out) valid_out[j] = valid[j];
  }
  if (near_ties_out) *near_ties_out = near;
  return BD_OK;
}

extern "C" bd_status rl_select(int32_t n, int32_t m, int32_t ref_index, const uint8_t* correct,
                               const uint8_t* prompt_mask, const double* cost, double alpha,
                               double delta, int32_t method, const int32_t* order, int32_t* V_out,
                               double* p_out, uint8_t* valid_out, int32_t* selected_out) {
  if (!check_common("rl_select", n, m, ref_index, correct, cost, alpha, delta, method, order))
    return BD_EINVAL;
  if (!selected_out) {
    bd::set_error("rl_select: selected_out is NULL");
    return BD_EINVAL;
  }
  std::vector<uint64_t> mask;
  int64_t n_eff = n;
  if (prompt_mask) {
    mask = pack_mask(prompt_mask, n, false);
    n_eff = 0;
    for (int i = 0; i < n; ++i) n_eff += prompt_mask[i] != 0;
    if (n_eff == 0) {
      bd::set_error("rl_select: the prompt mask selects no prompt");
      return BD_EINVAL;
    }
  }
  ViolBits vb(m, n, ref_index, correct);
  std::vector<int64_t> V(m);
  std::vector<long double> p(m);
  for (int j = 0; j < m; ++j) {
    V[j] = vb.count(j, prompt_mask ? mask.data() : nullptr);
    p[j] = binom_cdf(n_eff, alpha, V[j]);
  }
  std::vector<uint8_t> valid(m);
  valid_set(method, m, p.data(), V.data(), n_eff, alpha, delta, order, valid.data(), nullptr);
  *selected_out = deploy(m, cost, valid.data(), ref_index);
  for (int j = 0; j < m; ++j) {
    if (V_out) V_out[j] = (int32_t)V[j];
    if (p_out) p_out[j] = (double)p[j];
    if (valid_out) valid_out[j] = valid[j];
  }
  return BD_OK;
}

extern "C" bd_status rl_alpha_sweep(int32_t n, int32_t m, int32_t ref_index, const uint8_t* correct,
                                    const double* cost, const double* alphas, int32_t n_alpha,
                                    double delta, int32_t method, const int32_t* order,
                                    int32_t* selected_out, int32_t* n_valid_out,
                                    double* alpha_hat_out) {
  if (n_alpha < 1 || !alphas || !selected_out) {
    bd::set_error("rl_alpha_sweep: need n_alpha >= 1, alphas and selected_out");
    return BD_EINVAL;
  }
  for (int k = 0; k < n_alpha; ++k)
    if (!check_common("rl_alpha_sweep", n, m, ref_index, correct, cost, alphas[k], delta, method, order))
      return BD_EINVAL;
  ViolBits vb(m, n, ref_index, correct);
  std::vector<int64_t> V(m);
  for (int j = 0; j < m; ++j) V[j] = vb.count(j, nullptr);
  double hat = NAN;
  std::vector<long double> p(m);
  std::vector<uint8_t> valid(m);
  for (int k = 0; k < n_alpha; ++k) {
    for (int j = 0; j < m; ++j) p[j] = binom_cdf(n, alphas[k], V[j]);
    valid_set(method, m, p.data(), V.data(), n, alphas[k], delta, order, valid.data(), nullptr);
    selected_out[k] = deploy(m, cost, valid.data(), ref_index);
    int nv = 0;
    bool gain = false;
    for (int j = 0; j < m; ++j) {
      nv += valid[j];
      gain |= valid[j] && cost[j] > cost[ref_index];
    }
    if (n_valid_out) n_valid_out[k] = nv;
    if (gain && !(hat <= alphas[k])) hat = alphas[k];
  }
  if (alpha_hat_out) *alpha_hat_out = hat;
  return BD_OK;
}

extern "C" bd_status rl_split_exceedance(int32_t n, int32_t m, int32_t ref_index,
                                         const uint8_t* correct, const double* cost, double alpha,
                                         double delta, int32_t method, const int32_t* order,
                                         int32_t n_splits, const uint8_t* cal_masks,
                                         int32_t* deployed_out, int32_t* test_viol_out,
                                         int32_t* counts_out, double* gain_sum_out) {
  if (!check_common("rl_split_exceedance", n, m, ref_index, correct, cost, alpha, delta, method, order))
    return BD_EINVAL;
  if (n_splits < 1 || !cal_masks) {
    bd::set_error("rl_split_exceedance: need n_splits >= 1 and cal_masks");
    return BD_EINVAL;
  }
  std::vector<int64_t> n_cal(n_splits, 0);
  for (int s = 0; s < n_splits; ++s) {
    for (int i = 0; i < n; ++i) n_cal[s] += cal_masks[(size_t)s * n + i] != 0;
    if (n_cal[s] == 0 || n_cal[s] == n) {
      bd::set_error("rl_split_exceedance: every split needs calibration and test prompts");
      return BD_EINVAL;
    }
  }
  const ViolBits vb(m, n, ref_index, correct);
  std::vector<int64_t> V_all(m);
  for (int j = 0; j < m; ++j) V_all[j] = vb.count(j, nullptr);
  std::vector<int32_t> dep(n_splits), tv(n_splits);
  std::vector<uint8_t> ex_t(n_splits), ex_p(n_splits), fw_t(n_splits), fw_p(n_splits);
  const int nt = (int)std::min<unsigned>(std::max(1u, std::thread::hardware_concurrency()), 64u);
  std::vector<PvalCache> caches(nt, PvalCache(alpha));
  parallel_for(n_splits, [&](int s, int t) {
    const std::vector<uint64_t> cal = pack_mask(cal_masks + (size_t)s * n, n, false);
    const std::vector<uint64_t> test = pack_mask(cal_masks + (size_t)s * n, n, true);
    const int64_t n_test = n - n_cal[s];
    std::vector<int64_t> V(m), Vt(m);
    std::vector<long double> p(m);
    std::vector<uint8_t> valid(m);
    for (int j = 0; j < m; ++j) {
      V[j] = vb.count(j, cal.data());
      Vt[j] = vb.count(j, test.data());
      p[j] = caches[t](n_cal[s], V[j]);
    }
    valid_set(method, m, p.data(), V.data(), n_cal[s], alpha, delta, order, valid.data(), nullptr);
    const int d = deploy(m, cost, valid.data(), ref_index);
    dep[s] = d;
    tv[s] = (int32_t)Vt[d];
    auto r_test = [&](int j) { return (double)Vt[j] / (double)n_test; };
    auto r_pool = [&](int j) { return (double)V_all[j] / (double)n; };
    ex_t[s] = r_test(d) > alpha;
    ex_p[s] = r_pool(d) > alpha;
    bool ft = false, fp = false;
    for (int j = 0; j < m; ++j) {
      ft |= valid[j] && r_test(j) > alpha;
      fp |= valid[j] && r_pool(j) > alpha;
    }
    fw_t[s] = ft;
    fw_p[s] = fp;
  });
  int32_t c[4] = {0, 0, 0, 0};
  double gain = 0.0;
  for (int s = 0; s < n_splits; ++s) {   // in split order, as a sequential sum
    c[0] += ex_t[s];
    c[1] += ex_p[s];
    c[2] += fw_t[s];
    c[3] += fw_p[s];
    gain += cost[dep[s]] / cost[ref_index] - 1.0;
    if (deployed_out) deployed_out[s] = dep[s];
    if (test_viol_out) test_viol_out[s] = tv[s];
  }
  if (counts_out) std::copy(c, c + 4, counts_out);
  if (gain_sum_out) *gain_sum_out = gain;
  return BD_OK;
}

extern "C" bd_status rl_monte_carlo(int32_t n, int32_t m, const double* true_risk, double alpha,
                                    double delta, int32_t method, const int32_t* order,
                                    int32_t trials, int32_t k, const double* u,
                                    int32_t* false_trials_out, int32_t* valid_counts_out) {
  // the cost vector is not used; any non-NULL pointer passes the common check
  const double dummy = 0.0;
  if (!check_common("rl_monte_carlo", n, m, 0, true_risk, &dummy, alpha, delta, method, order))
    return BD_EINVAL;
  if (trials < 1 || !u || !false_trials_out || (k != 1 && k != m)) {
    bd::set_error("rl_monte_carlo: need trials >= 1, k = 1 or m, u and false_trials_out");
    return BD_EINVAL;
  }
  std::vector<uint8_t> valid_all((size_t)trials * m), false_t(trials);
  const int nt = (int)std::min<unsigned>(std::max(1u, std::thread::hardware_concurrency()), 64u);
  std::vector<PvalCache> caches(nt, PvalCache(alpha));
  parallel_for(trials, [&](int tr, int t) {
    std::vector<int64_t> V(m);
    std::vector<long double> p(m);
    uint8_t* valid = &valid_all[(size_t)tr * m];
    for (int j = 0; j < m; ++j) {
      const double* row = u + ((size_t)tr * k + (k == 1 ? 0 : j)) * n;
      int64_t c = 0;
      for (int i = 0; i < n; ++i) c += row[i] < true_risk[j];
      V[j] = c;
      p[j] = caches[t](n, c);
    }
    valid_set(method, m, p.data(), V.data(), n, alpha, delta, order, valid, nullptr);
    bool f = false;
    for (int j = 0; j < m; ++j) f |= valid[j] && true_risk[j] > alpha;
    false_t[tr] = f;
  });
  int32_t ft = 0;
  for (int tr = 0; tr < trials; ++tr) ft += false_t[tr];
  *false_trials_out = ft;
  if (valid_counts_out)
    for (int j = 0; j < m; ++j) {
      int32_t c = 0;
      for (int tr = 0; tr < trials; ++tr) c += valid_all[(size_t)tr * m + j];
      valid_counts_out[j] = c;
    }
  return BD_OK;
}
