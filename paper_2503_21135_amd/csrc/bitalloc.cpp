// bitalloc.cpp -- offline expert-level bit allocation on the host.
//
// Sec. III-B, Eq. (1): expert significance of one dataset from per-token
// significance and the router's top-K choices.  Sec. IV-A, Alg. 1: fuzzy
// c-means over the experts' significance, one precision per cluster from the
// most to the least significant, and the low-precision-first rule for experts
// that sit in the overlap of clusters.  This runs once per dataset on a few
// hundred numbers, so it is plain host code; its output is the per-expert
// bit-width list that moe_quant_pack and moe_requant_channels take.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <numeric>
#include <vector>

#include "moe_quant.h"

extern "C" int moe_expert_significance(const float* sig, const int32_t* topk_ids, int32_t T,
                                       int32_t k, int32_t E, double* s_exp, double* share) {
  if (T < 0 || k < 1 || k > MOE_MAX_TOPK || E < 1 || E > MOE_MAX_EXPERTS) return MOE_ERR_ARG;
  if (!s_exp || (T > 0 && (!sig || !topk_ids))) return MOE_ERR_ARG;
  for (int64_t i = 0; i < static_cast<int64_t>(T) * k; i++)
    if (topk_ids[i] < 0 || topk_ids[i] >= E) return MOE_ERR_ARG;
  for (int32_t i = 0; i < T; i++)
    if (!(sig[i] >= 0.0f) || !std::isfinite(sig[i])) return MOE_ERR_ARG;
  std::vector<double> num(E, 0.0);
  std::vector<int64_t> cnt(E, 0);
  double total = 0.0;
  // tokens in order, so each expert's sum adds its tokens in ascending order
  for (int32_t i = 0; i < T; i++) {
    const int32_t* row = topk_ids + static_cast<int64_t>(i) * k;
    const double s = static_cast<double>(sig[i]);
    total += s;
    for (int a = 0; a < k; a++) {
      bool dup = false;
      for (int b = 0; b < a; b++) dup = dup || row[b] == row[a];
      if (dup) continue;  // an expert counts once per token
      num[row[a]] += s;
      cnt[row[a]]++;
    }
  }
  for (int e = 0; e < E; e++) {
    s_exp[e] = total > 0.0 ? num[e] / total : 0.0;
    if (share) share[e] = T > 0 ? static_cast<double>(cnt[e]) / T : 0.0;
  }
  return MOE_OK;
}

extern "C" int moe_allocate_bits(const double* x, const double* share, int32_t n,
                                 const int32_t* levels, int32_t c, double m, double eps,
                                 int32_t max_iter, double alpha, int32_t* bits, double* V,
                                 double* U, int32_t* rounds) {
  if (n < 1 || c < 1 || c > 8 || !x || !share || !levels || !bits) return MOE_ERR_ARG;
  if (!(m > 1.0) || !std::isfinite(m) || !(eps > 0.0) || max_iter < 1 || !std::isfinite(alpha))
    return MOE_ERR_ARG;
  for (int k = 0; k < c; k++)
    if (levels[k] < 1 || levels[k] > 8) return MOE_ERR_BITS;
  double tot = 0.0;
  for (int i = 0; i < n; i++) {
    if (!std::isfinite(x[i]) || !(share[i] >= 0.0) || !std::isfinite(share[i])) return MOE_ERR_ARG;
    tot += share[i];
  }

  // Initial scores: experts by ascending significance (ties by index), cut
  // into c runs of equal token share; an expert joins the run that holds the
  // midpoint of its own share.
  std::vector<int> order(n);
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return x[a] < x[b]; });
  std::vector<double> u(static_cast<size_t>(n) * c, 0.0), un(u.size(), 0.0), v(c, 0.0);
  double run = 0.0;
  for (int r = 0; r < n; r++) {
    const int i = order[r];
    const double mid = tot > 0.0 ? (run + share[i] / 2.0) / tot : (r + 0.5) / n;
    const int k = std::min(static_cast<int>(mid * c), c - 1);
    u[static_cast<size_t>(i) * c + k] = 1.0;
    run += share[i];
  }

  const double p = 2.0 / (m - 1.0);
  std::vector<double> d(c);
  int round = 0;
  for (;;) {
    round++;
    for (int k = 0; k < c; k++) {  // centers: membership^m weighted means
      double sw = 0.0, swx = 0.0;
      for (int i = 0; i < n; i++) {
        const double w = std::pow(u[static_cast<size_t>(i) * c + k], m);
        sw += w;
        swx += w * x[i];
      }
      v[k] = sw > 0.0 ? swx / sw : 0.0;
    }
    double delta2 = 0.0;
    for (int i = 0; i < n; i++) {  // memberships from the distances to the centers
      double* ui = &un[static_cast<size_t>(i) * c];
      int zeros = 0;
      for (int k = 0; k < c; k++) {
        d[k] = std::fabs(x[i] - v[k]);
        zeros += d[k] == 0.0;
      }
      for (int k = 0; k < c; k++) {
        if (zeros) {
          ui[k] = d[k] == 0.0 ? 1.0 / zeros : 0.0;
        } else {
          double s = 0.0;
          for (int j = 0; j < c; j++) s += std::pow(d[k] / d[j], p);
          ui[k] = 1.0 / s;
        }
        const double dd = ui[k] - u[static_cast<size_t>(i) * c + k];
        delta2 += dd * dd;
      }
    }
    u.swap(un);
    if (std::sqrt(delta2) < eps || round >= max_iter) break;
  }

  // Cluster precision: the largest center takes levels[0], and so on down.
  std::vector<int> rank(c);
  std::iota(rank.begin(), rank.end(), 0);
  std::stable_sort(rank.begin(), rank.end(), [&](int a, int b) { return v[a] > v[b]; });
  std::vector<int32_t> cl(c);
  for (int r = 0; r < c; r++) cl[rank[r]] = levels[r];
  // Low-precision-first: the lowest precision among the clusters whose
  // membership reaches alpha; else the cluster of largest membership.
  for (int i = 0; i < n; i++) {
    const double* ui = &u[static_cast<size_t>(i) * c];
    int32_t b = 0;
    for (int k = 0; k < c; k++)
      if (ui[k] >= alpha && (b == 0 || cl[k] < b)) b = cl[k];
    if (b == 0) b = cl[std::max_element(ui, ui + c) - ui];
    bits[i] = b;
  }
  if (V) std::copy(v.begin(), v.end(), V);
  if (U) std::copy(u.begin(), u.end(), U);
  if (rounds) *rounds = round;
  return MOE_OK;
}
