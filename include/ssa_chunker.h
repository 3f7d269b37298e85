/*
 * ssa_chunker.h -- SlidingChunker and TimeToBudget (SlidingServe Sec. 3.4,
 * Alg. 1, Eq. 14-16), on the batch latency predictor (ssa_predictor.h).
 *
 * Host-only C ABI in libssa.so.  Given the decode requests D, the prefill
 * requests P in the order the priority sorter put them, the server's maximum
 * budget B and the latency bounds of the current and the next iteration of the
 * window (T_cur, T_next; Eq. 14-15), choose this iteration's token budget b and
 * the chunk each prefill request gets.
 *
 * Batch forming (the paper's BatchForwarder, the serving engine's token allocation): every
 * decode request gets one token; the rest of the budget goes to the prefill
 * requests in order, each taking min(its remaining prompt tokens, what is left).
 * The formed batch's features (Tab. 1) and scene (Eq. 3) feed the predictor;
 * a request given one token counts as a decode row there (Eq. 2), and one given
 * none is not in the batch; an empty batch is predicted to take no time.
 * Budgets below |D| are taken as |D| (the decodes always run) and budgets
 * above B as B.
 *
 * TimeToBudget(T): the largest b in [|D|, B] whose formed batch the predictor
 * puts at or below T, by binary search (exact when the prediction does not
 * decrease with b; |D| if even that exceeds T).
 *
 * SlidingChunker (Alg. 1): B_cur = TimeToBudget(T_cur), B_next =
 * TimeToBudget(T_next), B_sum = B_cur + B_next, and the budget b in
 * [|D|, min(B, B_cur)] that minimises the window cost pred(b) + pred(B_sum - b)
 * (Eq. 16), ties to the larger budget.  The paper approximates this argmin with
 * a discrete ternary search; here it is exact: the window cost is piecewise
 * quadratic in b (between the budgets where the partially served prefill
 * request changes, where its chunk crosses 0, 1 or 2 tokens or the largest full
 * chunk, and where form's clamps act, every Tab. 1 feature is a polynomial of
 * degree <= 2 in b and the scene is fixed), so each piece's minimum lies at an
 * end or next to the vertex of its quadratic, and only those budgets are
 * scored.  The upper bound is capped by B_cur: a budget beyond it would break
 * this iteration's own bound T_cur.
 *
 * All calls return 0 or a negative SSA_ERR_* code (ssa.h) and write nothing on
 * an error; they allocate nothing.
 */
#ifndef SSA_CHUNKER_H
#define SSA_CHUNKER_H

#include <stdint.h>

#include "ssa_predictor.h"

#ifdef __cplusplus
extern "C" {
#endif

/* A prefill request: tokens already cached (u) and prompt tokens still to prefill. */
typedef struct ssa_prefill_request {
  int32_t cached;
  int32_t remaining;
} ssa_prefill_request;

/*
 * The batch that budget b forms: chunk[k] = tokens given to prefill[k]
 * (n_prefill entries, caller's buffer), its features x[0..6] and scene.
 * Errors: SSA_ERR_NULL (decode_ctx with n_decode > 0, prefill with
 * n_prefill > 0, chunk with n_prefill > 0, x, scene); SSA_ERR_ARG (negative
 * counts, lengths or budgets).
 */
int ssa_form_batch(const int32_t* decode_ctx, int32_t n_decode, const ssa_prefill_request* prefill,
                   int32_t n_prefill, int32_t budget, int32_t max_budget, int32_t* chunk, double* x,
                   int32_t* scene);

/*
 * TimeToBudget: the largest budget in [n_decode, max_budget] whose formed
 * batch the predictor puts at or below t_limit (see above).  Errors: those of
 * ssa_form_batch and ssa_predictor_predict; SSA_ERR_ARG if max_budget < n_decode.
 */
int ssa_time_to_budget(const ssa_predictor* pred, const int32_t* decode_ctx, int32_t n_decode,
                       const ssa_prefill_request* prefill, int32_t n_prefill, int32_t max_budget,
                       double t_limit, int32_t* budget);

/*
 * SlidingChunker (Alg. 1).  Returns the budget, the chunk of every prefill
 * request (chunk, n_prefill entries) and the predicted latency of this
 * iteration's batch (t_pred; may be NULL).  Errors: as ssa_time_to_budget.
 */
int ssa_sliding_chunker(const ssa_predictor* pred, const int32_t* decode_ctx, int32_t n_decode,
                        const ssa_prefill_request* prefill, int32_t n_prefill, int32_t max_budget,
                        double t_cur, double t_next, int32_t* budget, int32_t* chunk,
                        double* t_pred);

#ifdef __cplusplus
}
#endif

#endif /* SSA_CHUNKER_H */
