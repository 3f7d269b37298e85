/*
 * ssa_constructor.h -- Multi-Level Priority Sorter, Violation Checker and
 * BatchConstructor (SlidingServe Sec. 3.3, Eq. 6-13; Sec. 3.5, Eq. 17-22,
 * Alg. 2), on the batch latency predictor (ssa_predictor.h) and the batch
 * forming and TimeToBudget of ssa_chunker.h.
 *
 * Host-only C ABI in libssa.so.  Times (slacks, predictions) are in the unit
 * the predictor was fitted in; throughput is tokens per that unit.
 *
 * Priority sort (Eq. 6-13).  For a prefilling or waiting request i with
 * remaining prompt tokens r_i, TTFT slack s_i and safeguard flag g_i:
 *   u_i = r_i / (rho * max(s_i, eps))   (urgency, Eq. 10; rho = recent throughput)
 *   e_i = [u_i > alpha]                 (urgent, Eq. 11)
 *   key K_i = (1 - g_i, 1 - e_i, r_i), sorted ascending (Eq. 12-13); equal keys
 *   keep their input order (arrival order).
 * alpha and eps are the caller's (the paper does not give them).
 *
 * BatchConstructor (Alg. 2), on candidates in priority order:
 *   1. T_full = predicted latency of the batch the full budget B forms.
 *   2. Violation check: the risky requests are those with s_j < T_full.  None:
 *      outcome SSA_CONSTRUCT_NO_RISK (keep the SlidingChunker's batch).
 *   3. C = the candidates by increasing (s_j, r_j) (the printed "sort C" names a
 *      set never defined; read as the candidates), and every risky request in
 *      that order is an anchor a:
 *        B_a = TimeToBudget(s_a) (the budget predicted within the anchor's
 *        slack), C_a = min(B, B_a) - |D| (Eq. 17); infeasible if C_a <= 0 or r_a > C_a;
 *        S_a = the candidates with s_j >= s_a (a included);
 *        v_j = 1 / (s'_j / sum_{S_a} s' + r_j / sum_{S_a} r) with s' = max(s, eps)
 *        (Eq. 18; slacks of late requests are negative, hence the clamp);
 *        Y = 0/1 knapsack over S_a minus a (Eq. 19): most total value within capacity
 *        C_a - r_a, weights r_j (dynamic programming over integer capacity;
 *        items in C order, a later item replaces an earlier choice only when
 *        strictly better), plus a (Eq. 20);
 *        the comparer keeps Y when (|Y|, sum v, sum r) is lexicographically
 *        larger than the best so far (Eq. 21), so the first of equal ones stays.
 *   4. Outcome SSA_CONSTRUCT_BATCH with budget |D| + sum_{Y*} r_j, every chosen
 *      request taking all its remaining tokens (Eq. 22); or, if no anchor was
 *      feasible, SSA_CONSTRUCT_NO_ANCHOR (the printed algorithm would return
 *      the decodes alone; the caller keeps the SlidingChunker's batch).
 *
 * All calls return 0 or a negative SSA_ERR_* code (ssa.h) and write nothing on
 * an error.
 */
#ifndef SSA_CONSTRUCTOR_H
#define SSA_CONSTRUCTOR_H

#include <stdint.h>

#include "ssa_chunker.h"

#ifdef __cplusplus
extern "C" {
#endif

/* A prefilling or waiting request. */
typedef struct ssa_candidate {
  int32_t cached;    /* tokens already in the cache (u) */
  int32_t remaining; /* prompt tokens still to prefill, r = p - c(t) */
  double slack;      /* TTFT slack s = a + L_ttft - t */
  int32_t safeguard; /* g: 1 = protected */
  int32_t reserved;
} ssa_candidate;

enum { SSA_CONSTRUCT_NO_RISK = 0, SSA_CONSTRUCT_NO_ANCHOR = 1, SSA_CONSTRUCT_BATCH = 2 };

/*
 * Priority order (Eq. 12-13): order[k] = index of the k-th candidate.
 * Errors: SSA_ERR_NULL (cand or order with n > 0); SSA_ERR_ARG (n < 0,
 * throughput <= 0, eps <= 0, a non-finite slack, alpha or throughput, negative
 * remaining).
 */
int ssa_priority_sort(const ssa_candidate* cand, int32_t n, double throughput, double alpha,
                      double eps, int32_t* order);

/*
 * Alg. 2 on candidates in priority order.  Outputs: outcome (SSA_CONSTRUCT_*);
 * budget and take[k] (tokens given to candidate k: its remaining tokens or 0)
 * when the outcome is SSA_CONSTRUCT_BATCH, else unchanged; t_full (may be
 * NULL).  Capacity: max_budget up to 1 << 20.  Errors: those of
 * ssa_time_to_budget; SSA_ERR_NULL (pred, outcome, budget, take with n > 0);
 * SSA_ERR_ARG (eps <= 0, max_budget above 1 << 20, non-finite slacks, negative
 * lengths).
 */
int ssa_batch_constructor(const ssa_predictor* pred, const int32_t* decode_ctx, int32_t n_decode,
                          const ssa_candidate* cand, int32_t n, int32_t max_budget, double eps,
                          int32_t* outcome, int32_t* budget, int32_t* take, double* t_full);

#ifdef __cplusplus
}
#endif

#endif /* SSA_CONSTRUCTOR_H */
