// SlidingChunker and TimeToBudget (SlidingServe Sec. 3.4, Alg. 1, Eq. 14-16)
// over the batch latency predictor.  Host code; the contract, including the
// readings where the printed algorithm is silent, is in include/ssa_chunker.h.

#include <algorithm>
#include <cstdint>

#include "../../include/ssa_chunker.h"

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

}  // namespace

extern "C" {

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
  const int64_t b_sum = b_cur + b_next;
  // window cost of budget b: this iteration plus the next one with the rest
  auto cost = [&](int64_t b, double* c) {
    double t1 = 0.0, t2 = 0.0;
    int r = pred(pred_model, q, b, &t1);
    if (!r) r = pred(pred_model, q, b_sum - b, &t2);
    *c = t1 + t2;
    return r;
  };
  int64_t l = n_decode, r = std::min<int64_t>(max_budget, b_cur);
  const int64_t l0 = l, r0 = r;
  while (r - l > 30) {
    const int64_t m1 = l + (r - l) / 3, m2 = r - (r - l) / 3;
    double c1, c2;
    if ((rc = cost(m1, &c1)) || (rc = cost(m2, &c2))) return rc;
    if (c1 <= c2)
      r = m2 - 1;
    else
      l = m1 + 1;
  }
  const int64_t cand[3] = {l0, r0, l + (r - l) / 2};
  int64_t best = l0;
  double best_cost = 0.0;
  bool have = false;
  for (int64_t b : cand) {
    double c;
    if ((rc = cost(b, &c))) return rc;
    if (!have || c < best_cost || (c == best_cost && b > best)) {
      best = b;
      best_cost = c;
      have = true;
    }
  }
  double x[SSA_PRED_FEATURES];
  int32_t scene = 0;
  form(q, best, chunk, x, &scene);
  if (t_pred && (rc = pred(pred_model, q, best, t_pred))) return rc;
  *budget = (int32_t)best;
  return SSA_OK;
}

}  // extern "C"
