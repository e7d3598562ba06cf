// Locality score of the code cache's entries and the residency it implies
// (Sec. 4.1, Eq. 3; App. B.1, Eq. 8-10; the update step of Alg. 1).  Host
// code: it decides which segments stay in device memory; fcg_lib_offload /
// fcg_lib_reload move them.
//
//   l(f) = (1 - l_curr(f)) (alpha l_freq(f) + beta sum_j l_asso(j | f) + gamma l_sema(f)) + l_curr(f)
//   l_freq(f) = count(f) / max_j count(j), l_asso(j | f) = cooccur(f, j) / count(f),
//   l_sema(f) = PPL(f) / max_j PPL(j)
//
// Statistics cover the last `window` execution traces (one per task);
// cooccur(f, j) counts the calls of j that immediately follow a call of f in
// one trace; l_curr(f) = 1 iff f occurs in the latest trace; a component with
// a zero denominator is 0.
#include <algorithm>
#include <cmath>
#include <deque>
#include <new>
#include <numeric>
#include <string>
#include <vector>

#include "errors.hpp"
#include "locality.hpp"

struct fcg_locality {
  int32_t n, window;
  double alpha, beta, gamma;
  std::deque<std::vector<int32_t>> traces;
  std::vector<double> ppl;
};

namespace {

// the scores in the order of the formula above
void compute_scores(const fcg_locality& L, double* out) {
  const int32_t n = L.n;
  std::vector<int64_t> count(n, 0);
  for (const auto& t : L.traces)
    for (int32_t f : t) ++count[f];
  const int64_t top = *std::max_element(count.begin(), count.end());
  const double ptop = *std::max_element(L.ppl.begin(), L.ppl.end());
  std::vector<double> cur(n, 0.0);
  if (!L.traces.empty())
    for (int32_t f : L.traces.back()) cur[f] = 1.0;
  for (int32_t f = 0; f < n; ++f) {
    const double freq = top > 0 ? (double)count[f] / (double)top : 0.0;
    // sum_j cooccur(f, j) / count(f), term by term as in the definition
    double asso = 0.0;
    if (count[f] > 0) {
      std::vector<int64_t> row(n, 0);
      for (const auto& t : L.traces)
        for (size_t i = 0; i + 1 < t.size(); ++i)
          if (t[i] == f) ++row[t[i + 1]];
      for (int32_t j = 0; j < n; ++j) asso += (double)row[j] / (double)count[f];
    }
    const double sema = ptop > 0 ? L.ppl[f] / ptop : 0.0;
    const double mix = L.alpha * freq + L.beta * asso + L.gamma * sema;
    out[f] = (1.0 - cur[f]) * mix + cur[f];
  }
}

}  // namespace

// Residency under a budget (the update step of Alg. 1): entries that must stay
// (pinned) first, their cost counted; then, in descending score (ties:
// ascending id), an entry is kept when its cost still fits.  With tau > 0 the
// entries whose perplexity is below tau come after all the others (the
// perplexity-based eviction threshold of the hyperparameter table: code the
// model already predicts well leaves the device tier first).
fcg_status fcg::locality_residency(const fcg_locality* L, int64_t budget, const int64_t* cost, double tau,
                                   const uint8_t* pinned, uint8_t* resident) {
  if (!L || !cost || !resident) return fcg::report(FCG_EINVAL, "null argument");
  if (budget < 0) return fcg::report(FCG_EINVAL, "negative budget");
  if (!(tau >= 0)) return fcg::report(FCG_EINVAL, "the perplexity threshold must be >= 0");
  for (int32_t f = 0; f < L->n; ++f)
    if (cost[f] < 0) return fcg::report(FCG_EINVAL, "negative cost");
  std::vector<double> s(L->n);
  compute_scores(*L, s.data());
  std::vector<int32_t> order(L->n);
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) { return s[a] > s[b]; });
  int64_t used = 0;
  for (int32_t f = 0; f < L->n; ++f) {
    resident[f] = pinned && pinned[f];
    if (resident[f]) used += cost[f];
  }
  for (int pass = 0; pass < (tau > 0 ? 2 : 1); ++pass)
    for (int32_t f : order) {
      if (resident[f]) continue;
      if (tau > 0 && (L->ppl[f] >= tau) != (pass == 0)) continue;
      if (used + cost[f] <= budget) {
        resident[f] = 1;
        used += cost[f];
      }
    }
  return FCG_OK;
}

int32_t fcg::locality_size(const fcg_locality* L) { return L ? L->n : 0; }

extern "C" {

fcg_status fcg_locality_create(int32_t n_funcs, int32_t window, double alpha, double beta, double gamma,
                               fcg_locality** out) {
  if (!out) return fcg::report(FCG_EINVAL, "null output handle");
  if (n_funcs < 1 || window < 1) return fcg::report(FCG_EINVAL, "n_funcs and window must be >= 1");
  if (!(alpha >= 0 && beta >= 0 && gamma >= 0) || std::fabs(alpha + beta + gamma - 1.0) > 1e-9)
    return fcg::report(FCG_EINVAL, "alpha, beta, gamma must be >= 0 and sum to 1");
  fcg_locality* L = new (std::nothrow) fcg_locality{n_funcs, window, alpha, beta, gamma, {}, {}};
  if (!L) return fcg::report(FCG_ENOMEM, "host allocation");
  L->ppl.assign(n_funcs, 0.0);
  *out = L;
  return FCG_OK;
}

fcg_status fcg_locality_record(fcg_locality* L, int32_t n, const int32_t* func_ids) {
  if (!L) return fcg::report(FCG_EINVAL, "null handle");
  if (n < 0 || (n > 0 && !func_ids)) return fcg::report(FCG_EINVAL, "bad trace");
  for (int32_t i = 0; i < n; ++i)
    if (func_ids[i] < 0 || func_ids[i] >= L->n) return fcg::report(FCG_ERANGE, "function id out of range");
  L->traces.emplace_back(func_ids, func_ids + n);
  if ((int32_t)L->traces.size() > L->window) L->traces.pop_front();
  return FCG_OK;
}

fcg_status fcg_locality_set_ppl(fcg_locality* L, int32_t func, double ppl) {
  if (!L) return fcg::report(FCG_EINVAL, "null handle");
  if (func < 0 || func >= L->n) return fcg::report(FCG_ERANGE, "function id out of range");
  if (!(ppl >= 0)) return fcg::report(FCG_EINVAL, "perplexity must be >= 0");
  L->ppl[func] = ppl;
  return FCG_OK;
}

fcg_status fcg_locality_scores(const fcg_locality* L, double* scores) {
  if (!L || !scores) return fcg::report(FCG_EINVAL, "null argument");
  compute_scores(*L, scores);
  return FCG_OK;
}

fcg_status fcg_locality_residency(const fcg_locality* L, int64_t budget, const int64_t* cost, uint8_t* resident) {
  return fcg::locality_residency(L, budget, cost, 0.0, nullptr, resident);
}

fcg_status fcg_locality_destroy(fcg_locality* L) {
  delete L;
  return FCG_OK;
}

}  // extern "C"
