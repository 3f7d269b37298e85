// The scheduler around the attention path, on the batch latency predictor:
// SlidingChunker and TimeToBudget (SlidingServe Sec. 3.4, Alg. 1, Eq. 14-16),
// the Multi-Level Priority Sorter (Sec. 3.3, Eq. 6-13) and the BatchConstructor
// with its violation check (Sec. 3.5, Alg. 2, Eq. 17-22).  Host code; the
// contracts, including the readings where the paper is silent, are in
// include/ssa_chunker.h and include/ssa_constructor.h.

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <numeric>
#include <vector>

#include "../../include/ssa_chunker.h"
#include "../../include/ssa_constructor.h"

namespace {

struct Queue {
  const int32_t* dctx;
  int32_t nd;
  const ssa_prefill_request* pf;
  int32_t np;
  int64_t max_budget;
};

// The batch budget b forms (b clamped to [nd, max_budget]): chunks (if chunk
// is not NULL), Tab. 1 features and the Eq. 3 scene.  Every sum is of
// integers below 2^53, so the features are exact.
void form(const Queue& q, int64_t b, int32_t* chunk, double* x, int32_t* scene) {
  b = std::min(std::max(b, (int64_t)q.nd), q.max_budget);
  for (int j = 0; j < SSA_PRED_FEATURES; ++j) x[j] = 0.0;
  int64_t n_dec = 0, n_pre = 0;
  for (int32_t i = 0; i < q.nd; ++i) {  // decode rows: c = 1, u = context
    x[2] += q.dctx[i];
    x[3] += 1.0;
    x[4] += q.dctx[i];
    ++n_dec;
  }
  int64_t left = b - q.nd;
  for (int32_t k = 0; k < q.np; ++k) {
    const int64_t c = std::min<int64_t>(q.pf[k].remaining, left);
    left -= c;
    if (chunk) chunk[k] = (int32_t)c;
    if (c == 0) continue;
    const double u = q.pf[k].cached, cd = (double)c;
    x[2] += u;
    if (c <= 1) {  // Eq. 2: one new token is a decode row
      x[3] += 1.0;
      x[4] += u;
      ++n_dec;
    } else {
      x[0] += cd * (u + cd);
      x[1] += cd * cd;
      x[5] += cd;
      x[6] = std::max(x[6], cd);
      ++n_pre;
    }
  }
  *scene = n_dec + n_pre == 0 ? 0
           : n_pre == 0       ? SSA_SCENE_PURE_DECODE
           : n_dec == 0       ? SSA_SCENE_PURE_PREFILL
                              : SSA_SCENE_MIXED;
}

// Predicted latency of the batch budget b forms (0 for an empty batch).
int pred(const ssa_predictor* p, const Queue& q, int64_t b, double* t) {
  double x[SSA_PRED_FEATURES];
  int32_t scene = 0;
  form(q, b, nullptr, x, &scene);
  if (scene == 0) {
    *t = 0.0;
    return SSA_OK;
  }
  return ssa_predictor_predict(p, x, scene, t);
}

int check(const int32_t* dctx, int32_t nd, const ssa_prefill_request* pf, int32_t np,
          int32_t max_budget) {
  if ((nd > 0 && !dctx) || (np > 0 && !pf)) return SSA_ERR_NULL;
  if (nd < 0 || np < 0 || max_budget < 0) return SSA_ERR_ARG;
  for (int32_t i = 0; i < nd; ++i)
    if (dctx[i] < 0) return SSA_ERR_ARG;
  for (int32_t k = 0; k < np; ++k)
    if (pf[k].cached < 0 || pf[k].remaining < 0) return SSA_ERR_ARG;
  return SSA_OK;
}

// TimeToBudget: largest b in [nd, max_budget] predicted at or below t_limit.
int time_to_budget(const ssa_predictor* p, const Queue& q, double t_limit, int64_t* out) {
  int64_t lo = q.nd, hi = q.max_budget;
  double t;
  int rc = pred(p, q, lo, &t);
  if (rc) return rc;
  if (t > t_limit) {
    *out = lo;
    return SSA_OK;
  }
  while (lo < hi) {
    const int64_t mid = lo + (hi - lo + 1) / 2;
    rc = pred(p, q, mid, &t);
    if (rc) return rc;
    if (t <= t_limit)
      lo = mid;
    else
      hi = mid - 1;
  }
  *out = lo;
  return SSA_OK;
}

constexpr int64_t kMaxKnapsackCells = (int64_t)1 << 26;
constexpr int32_t kMaxConstructorBudget = 1 << 20;

int check_candidates(const ssa_candidate* c, int32_t n) {
  if (n > 0 && !c) return SSA_ERR_NULL;
  if (n < 0) return SSA_ERR_ARG;
  for (int32_t k = 0; k < n; ++k)
    if (c[k].cached < 0 || c[k].remaining < 0 || !std::isfinite(c[k].slack)) return SSA_ERR_ARG;
  return SSA_OK;
}

// 0/1 knapsack: the most total value within `cap` of the items (weights w,
// values v), items taken in order and a later item replacing an earlier
// choice only when strictly better.  Returns the chosen items' positions.
std::vector<int> knapsack(const std::vector<int64_t>& w, const std::vector<double>& v,
                          int64_t cap) {
  const size_t n = w.size();
  std::vector<double> best((size_t)cap + 1, 0.0);
  std::vector<uint8_t> keep(n * ((size_t)cap + 1), 0);
  for (size_t i = 0; i < n; ++i) {
    for (int64_t c = cap; c >= w[i]; --c) {
      const double cand = best[(size_t)(c - w[i])] + v[i];
      if (cand > best[(size_t)c]) {
        best[(size_t)c] = cand;
        keep[i * ((size_t)cap + 1) + (size_t)c] = 1;
      }
    }
  }
  std::vector<int> chosen;
  int64_t c = cap;
  for (size_t i = n; i-- > 0;) {
    if (keep[i * ((size_t)cap + 1) + (size_t)c]) {
      chosen.push_back((int)i);
      c -= w[i];
    }
  }
  std::reverse(chosen.begin(), chosen.end());
  return chosen;
}

// Eq. 16 over b in [q.nd, hi]: the budget minimising the window cost
// W(b) = pred(b) + pred(b_sum - b), ties to the larger budget.
//
// W is piecewise quadratic in b.  form() hands the budget left after the
// decodes to the prefill requests in order, so exactly one request is
// partially served at any budget and its chunk c grows by one per token.
// While that request is fixed and c stays on one side of the thresholds
// 0, 1, 2 (not in the batch / decode row / prefill row, Eq. 2) and of the
// largest full chunk (where x7 = max c switches), every Tab. 1 feature is a
// polynomial of degree <= 2 in c (x1 = sum c(u + c), x2 = sum c^2) and the
// scene is fixed, so pred is a fixed quadratic.  The same holds for the
// second term in b_sum - b, and for the clamps of form() at |D| and B.  The
// cuts between such pieces are collected below; on every piece the minimum
// of the quadratic is at an end or next to its vertex, found from three
// samples.  Every candidate is then scored with the real prediction, so the
// pick is the exact minimiser up to the rounding of pred itself.
int window_argmin(const ssa_predictor* p, const Queue& q, int64_t b_sum, int64_t hi,
                  int64_t* out) {
  const int64_t lo = q.nd;
  hi = std::max(hi, lo);
  // cuts in the budget domain of one pred() term: budget values where a new
  // piece starts
  std::vector<int64_t> starts{q.nd, q.nd + 1, q.max_budget, q.max_budget + 1};
  int64_t before = 0, largest_full = 0;  // tokens of the requests served fully; their max chunk
  for (int32_t k = 0; k < q.np; ++k) {
    const int64_t r = q.pf[k].remaining, s0 = q.nd + before;
    for (int64_t c : {(int64_t)0, (int64_t)1, (int64_t)2, largest_full, largest_full + 1, r, r + 1})
      if (c >= 0 && c <= r + 1) starts.push_back(s0 + c);
    before += r;
    if (r > 1) largest_full = std::max(largest_full, r);
  }
  std::vector<int64_t> cuts{lo, hi + 1};
  for (int64_t s : starts) {
    cuts.push_back(s);              // first term: b = s
    cuts.push_back(b_sum - s + 1);  // second term: b_sum - b < s from here on
    cuts.push_back(b_sum - s);
  }
  std::sort(cuts.begin(), cuts.end());
  cuts.erase(std::unique(cuts.begin(), cuts.end()), cuts.end());

  auto window = [&](int64_t b, double* w) {
    double t1 = 0.0, t2 = 0.0;
    int r = pred(p, q, b, &t1);
    if (!r) r = pred(p, q, b_sum - b, &t2);
    *w = t1 + t2;
    return r;
  };
  bool have = false;
  int64_t best = lo;
  double best_w = 0.0;
  auto consider = [&](int64_t b) {
    double w = 0.0;
    const int r = window(b, &w);
    if (!r && (!have || w < best_w || (w == best_w && b > best))) {
      have = true;
      best = b;
      best_w = w;
    }
    return r;
  };
  int rc = SSA_OK;
  for (size_t i = 0; i + 1 < cuts.size(); ++i) {
    const int64_t s = std::max(cuts[i], lo), e = std::min(cuts[i + 1] - 1, hi);
    if (s > e) continue;
    if ((rc = consider(s)) || (rc = consider(e))) return rc;
    if (e - s < 2) continue;
    const int64_t m = s + (e - s) / 2;
    double ws, wm, we;
    if ((rc = window(s, &ws)) || (rc = window(m, &wm)) || (rc = window(e, &we))) return rc;
    // quadratic through the three samples: curvature a, vertex v
    const double d1 = (wm - ws) / (double)(m - s), d2 = (we - wm) / (double)(e - m);
    const double a = (d2 - d1) / (double)(e - s);
    if (!(a > 0.0)) continue;  // linear or concave: the minimum is at an end
    const double v = 0.5 * ((double)(s + m) - d1 / a);
    if (!(v > (double)s && v < (double)e)) continue;
    const int64_t vf = (int64_t)std::floor(v);
    for (int64_t b = vf - 1; b <= vf + 2; ++b)
      if (b >= s && b <= e && (rc = consider(b))) return rc;
  }
  *out = best;
  return SSA_OK;
}

}  // namespace

extern "C" {

int ssa_priority_sort(const ssa_candidate* cand, int32_t n, double throughput, double alpha,
                      double eps, int32_t* order) {
  int rc = check_candidates(cand, n);
  if (rc) return rc;
  if (n > 0 && !order) return SSA_ERR_NULL;
  if (!(throughput > 0.0) || !(eps > 0.0) || !std::isfinite(throughput) ||
      !std::isfinite(alpha) || !std::isfinite(eps))
    return SSA_ERR_ARG;
  struct Key {
    int g, e;
    int32_t r;
  };
  std::vector<Key> key((size_t)n);
  for (int32_t k = 0; k < n; ++k) {
    const double u = (double)cand[k].remaining / (throughput * std::max(cand[k].slack, eps));
    key[(size_t)k] = Key{cand[k].safeguard ? 0 : 1, u > alpha ? 0 : 1, cand[k].remaining};
  }
  std::vector<int32_t> idx((size_t)n);
  std::iota(idx.begin(), idx.end(), 0);
  std::stable_sort(idx.begin(), idx.end(), [&](int32_t a, int32_t b) {
    const Key &x = key[(size_t)a], &y = key[(size_t)b];
    if (x.g != y.g) return x.g < y.g;
    if (x.e != y.e) return x.e < y.e;
    return x.r < y.r;
  });
  std::copy(idx.begin(), idx.end(), order);
  return SSA_OK;
}

int ssa_batch_constructor(const ssa_predictor* pred_model, const int32_t* decode_ctx,
                          int32_t n_decode, const ssa_candidate* cand, int32_t n,
                          int32_t max_budget, double eps, int32_t* outcome, int32_t* budget,
                          int32_t* take, double* t_full) {
  if (!pred_model || !outcome || !budget || (n > 0 && !take)) return SSA_ERR_NULL;
  int rc = check_candidates(cand, n);
  if (rc) return rc;
  if ((n_decode > 0 && !decode_ctx)) return SSA_ERR_NULL;
  if (n_decode < 0 || max_budget < n_decode || max_budget > kMaxConstructorBudget ||
      !(eps > 0.0) || !std::isfinite(eps))
    return SSA_ERR_ARG;
  for (int32_t i = 0; i < n_decode; ++i)
    if (decode_ctx[i] < 0) return SSA_ERR_ARG;
  std::vector<ssa_prefill_request> pf((size_t)n);
  for (int32_t k = 0; k < n; ++k) pf[(size_t)k] = ssa_prefill_request{cand[k].cached, cand[k].remaining};
  const Queue q{decode_ctx, n_decode, pf.data(), n, max_budget};
  // 1-2. the full batch's latency and the violation check
  double tf = 0.0;
  if ((rc = pred(pred_model, q, max_budget, &tf))) return rc;
  bool any_risk = false;
  for (int32_t k = 0; k < n; ++k) any_risk = any_risk || cand[k].slack < tf;
  if (!any_risk) {
    if (t_full) *t_full = tf;
    *outcome = SSA_CONSTRUCT_NO_RISK;
    return SSA_OK;
  }
  // 3. C: the candidates by increasing (slack, remaining), ties in priority order
  std::vector<int32_t> cord((size_t)n);
  std::iota(cord.begin(), cord.end(), 0);
  std::stable_sort(cord.begin(), cord.end(), [&](int32_t a, int32_t b) {
    if (cand[a].slack != cand[b].slack) return cand[a].slack < cand[b].slack;
    return cand[a].remaining < cand[b].remaining;
  });
  bool have = false;
  int64_t best_n = 0, best_r = 0;
  double best_v = 0.0;
  std::vector<uint8_t> best_set((size_t)n, 0);
  for (int32_t ai : cord) {
    const ssa_candidate& a = cand[ai];
    if (!(a.slack < tf)) continue;  // anchors: the risky requests
    int64_t b_a = 0;
    if ((rc = time_to_budget(pred_model, q, a.slack, &b_a))) return rc;
    const int64_t cap_a = std::min<int64_t>(max_budget, b_a) - n_decode;
    if (cap_a <= 0 || a.remaining > cap_a) continue;
    std::vector<int32_t> s_a;  // in C order, the anchor included
    double sum_s = 0.0;
    int64_t sum_r = 0;
    for (int32_t j : cord) {
      if (cand[j].slack >= a.slack) {
        s_a.push_back(j);
        sum_s += std::max(cand[j].slack, eps);
        sum_r += cand[j].remaining;
      }
    }
    std::vector<double> val(s_a.size());
    for (size_t k = 0; k < s_a.size(); ++k) {
      const ssa_candidate& c = cand[s_a[k]];
      const double rr = sum_r > 0 ? (double)c.remaining / (double)sum_r : 0.0;
      val[k] = 1.0 / (std::max(c.slack, eps) / sum_s + rr);
    }
    std::vector<int64_t> iw;
    std::vector<double> iv;
    std::vector<size_t> ipos;
    for (size_t k = 0; k < s_a.size(); ++k) {
      if (s_a[k] == ai) continue;
      iw.push_back(cand[s_a[k]].remaining);
      iv.push_back(val[k]);
      ipos.push_back(k);
    }
    const int64_t cap = cap_a - a.remaining;
    if ((int64_t)iw.size() * (cap + 1) > kMaxKnapsackCells) return SSA_ERR_ARG;
    std::vector<uint8_t> in_y(s_a.size(), 0);
    for (int p : knapsack(iw, iv, cap)) in_y[ipos[(size_t)p]] = 1;
    for (size_t k = 0; k < s_a.size(); ++k)
      if (s_a[k] == ai) in_y[k] = 1;
    int64_t yn = 0, yr = 0;
    double yv = 0.0;
    for (size_t k = 0; k < s_a.size(); ++k) {
      if (!in_y[k]) continue;
      ++yn;
      yv += val[k];
      yr += cand[s_a[k]].remaining;
    }
    const bool better = yn != best_n ? yn > best_n : (yv != best_v ? yv > best_v : yr > best_r);
    if (better) {
      have = true;
      best_n = yn;
      best_v = yv;
      best_r = yr;
      std::fill(best_set.begin(), best_set.end(), 0);
      for (size_t k = 0; k < s_a.size(); ++k)
        if (in_y[k]) best_set[(size_t)s_a[k]] = 1;
    }
  }
  if (t_full) *t_full = tf;
  if (!have) {
    *outcome = SSA_CONSTRUCT_NO_ANCHOR;
    return SSA_OK;
  }
  for (int32_t k = 0; k < n; ++k) take[k] = best_set[(size_t)k] ? cand[k].remaining : 0;
  *budget = (int32_t)(n_decode + best_r);
  *outcome = SSA_CONSTRUCT_BATCH;
  return SSA_OK;
}

int ssa_form_batch(const int32_t* decode_ctx, int32_t n_decode, const ssa_prefill_request* prefill,
                   int32_t n_prefill, int32_t budget, int32_t max_budget, int32_t* chunk, double* x,
                   int32_t* scene) {
  int rc = check(decode_ctx, n_decode, prefill, n_prefill, max_budget);
  if (rc) return rc;
  if (!x || !scene || (n_prefill > 0 && !chunk)) return SSA_ERR_NULL;
  if (budget < 0) return SSA_ERR_ARG;
  const Queue q{decode_ctx, n_decode, prefill, n_prefill, std::max(max_budget, n_decode)};
  form(q, budget, chunk, x, scene);
  return SSA_OK;
}

int ssa_time_to_budget(const ssa_predictor* pred_model, const int32_t* decode_ctx,
                       int32_t n_decode, const ssa_prefill_request* prefill, int32_t n_prefill,
                       int32_t max_budget, double t_limit, int32_t* budget) {
  if (!pred_model || !budget) return SSA_ERR_NULL;
  int rc = check(decode_ctx, n_decode, prefill, n_prefill, max_budget);
  if (rc) return rc;
  if (max_budget < n_decode) return SSA_ERR_ARG;
  const Queue q{decode_ctx, n_decode, prefill, n_prefill, max_budget};
  int64_t b = 0;
  rc = time_to_budget(pred_model, q, t_limit, &b);
  if (rc) return rc;
  *budget = (int32_t)b;
  return SSA_OK;
}

int ssa_sliding_chunker(const ssa_predictor* pred_model, const int32_t* decode_ctx,
                        int32_t n_decode, const ssa_prefill_request* prefill, int32_t n_prefill,
                        int32_t max_budget, double t_cur, double t_next, int32_t* budget,
                        int32_t* chunk, double* t_pred) {
  if (!pred_model || !budget || (n_prefill > 0 && !chunk)) return SSA_ERR_NULL;
  int rc = check(decode_ctx, n_decode, prefill, n_prefill, max_budget);
  if (rc) return rc;
  if (max_budget < n_decode) return SSA_ERR_ARG;
  const Queue q{decode_ctx, n_decode, prefill, n_prefill, max_budget};
  int64_t b_cur = 0, b_next = 0;
  if ((rc = time_to_budget(pred_model, q, t_cur, &b_cur))) return rc;
  if ((rc = time_to_budget(pred_model, q, t_next, &b_next))) return rc;
  int64_t best = 0;
  if ((rc = window_argmin(pred_model, q, b_cur + b_next, std::min<int64_t>(max_budget, b_cur),
                          &best)))
    return rc;
  double x[SSA_PRED_FEATURES];
  int32_t scene = 0;
  form(q, best, chunk, x, &scene);
  if (t_pred && (rc = pred(pred_model, q, best, t_pred))) return rc;
  *budget = (int32_t)best;
  return SSA_OK;
}

}  // extern "C"
