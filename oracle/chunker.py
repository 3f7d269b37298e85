"""CPU oracle of SlidingChunker and TimeToBudget (SlidingServe Sec. 3.4, Alg. 1,
Eq. 14-16).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, never by the library.  Plain
Python and numpy; it imports nothing from the library package.

What it computes:

* Batch forming (the paper's BatchForwarder): decodes take one token each; the
  rest of the budget goes to the prefill requests in their sorted order,
  min(remaining, left) each.  Budgets are clamped to [|D|, B].  The formed
  batch's features are Tab. 1 with Eq. 2's split (a request given one token is
  a decode row; one given none is not in the batch), and an empty batch takes
  no time.
* TimeToBudget(T): the largest budget predicted within T, by binary search over
  [|D|, B] (the paper inverts the predictor this way; exact whenever the
  prediction does not decrease with the budget, which a test checks against a
  scan of every budget).
* SlidingChunker: B_cur = TimeToBudget(T_cur), B_sum = B_cur +
  TimeToBudget(T_next), and the budget of Eq. 16, the argmin over b of
  pred(b) + pred(B_sum - b), taken here by evaluating every budget in
  [|D|, min(B, B_cur)] (the upper end capped by B_cur: a larger budget would
  break this iteration's own bound), ties to the larger budget.  The paper
  approximates the same argmin with a discrete ternary search.

The predictor is a dict {0: global, scene: model} of (b, w1..w7), evaluated as
b + w1 x1 + ... + w7 x7 in that order (Eq. 5), the scene's model first.
"""
from __future__ import annotations

import numpy as np

PURE_DECODE, PURE_PREFILL, MIXED = 1, 2, 3


def form_batch(decode_ctx, prefill, budget, max_budget):
    """(chunks, features x1..x7, scene) of the batch ``budget`` forms."""
    nd = len(decode_ctx)
    b = min(max(budget, nd), max(max_budget, nd))
    x = [0.0] * 7
    n_dec = n_pre = 0
    for u in decode_ctx:
        x[2] += u
        x[3] += 1.0
        x[4] += u
        n_dec += 1
    left = b - nd
    chunks = []
    for cached, remaining in prefill:
        c = min(remaining, left)
        left -= c
        chunks.append(c)
        if c == 0:
            continue
        x[2] += cached
        if c <= 1:
            x[3] += 1.0
            x[4] += cached
            n_dec += 1
        else:
            x[0] += float(c) * (cached + c)
            x[1] += float(c) * c
            x[5] += c
            x[6] = max(x[6], float(c))
            n_pre += 1
    if n_dec + n_pre == 0:
        scene = 0
    elif n_pre == 0:
        scene = PURE_DECODE
    elif n_dec == 0:
        scene = PURE_PREFILL
    else:
        scene = MIXED
    return chunks, x, scene


def predict(models, x, scene):
    if scene == 0:
        return 0.0
    coef = models.get(scene, models.get(0))
    t = coef[0]
    for j in range(7):
        t += coef[1 + j] * x[j]
    return t


def pred_budget(models, decode_ctx, prefill, b, max_budget):
    _, x, s = form_batch(decode_ctx, prefill, b, max_budget)
    return predict(models, x, s)


def time_to_budget(models, decode_ctx, prefill, max_budget, t_limit):
    lo, hi = len(decode_ctx), max_budget
    if pred_budget(models, decode_ctx, prefill, lo, max_budget) > t_limit:
        return lo
    while lo < hi:
        mid = lo + (hi - lo + 1) // 2
        if pred_budget(models, decode_ctx, prefill, mid, max_budget) <= t_limit:
            lo = mid
        else:
            hi = mid - 1
    return lo


def preds_over_budgets(models, decode_ctx, prefill, budgets, max_budget):
    """pred(b) for every budget in the integer array ``budgets``: the same
    batch forming, features and Eq. 5 sum as ``form_batch`` / ``predict``,
    elementwise over the budgets."""
    nd = len(decode_ctx)
    b = np.clip(np.asarray(budgets, dtype=np.int64), nd, max(max_budget, nd))
    n = b.shape[0]
    x = np.zeros((7, n), dtype=np.float64)
    dsum = float(sum(decode_ctx))
    x[2] += dsum
    x[3] += nd
    x[4] += dsum
    n_dec = np.full(n, nd, dtype=np.int64)
    n_pre = np.zeros(n, dtype=np.int64)
    left = b - nd
    for cached, remaining in prefill:
        c = np.minimum(remaining, left)
        left = left - c
        inb, dec, pre = c > 0, c == 1, c > 1
        x[2] += np.where(inb, cached, 0)
        x[3] += dec
        x[4] += np.where(dec, cached, 0)
        x[0] += np.where(pre, c * (cached + c), 0)
        x[1] += np.where(pre, c * c, 0)
        x[5] += np.where(pre, c, 0)
        x[6] = np.where(pre, np.maximum(x[6], c), x[6])
        n_dec += dec
        n_pre += pre
    scene = np.where(n_dec + n_pre == 0, 0,
                     np.where(n_pre == 0, PURE_DECODE, np.where(n_dec == 0, PURE_PREFILL, MIXED)))
    t = np.zeros(n, dtype=np.float64)
    for sc in (PURE_DECODE, PURE_PREFILL, MIXED):
        sel = scene == sc
        if not sel.any():
            continue
        coef = models.get(sc, models.get(0))
        ts = np.full(int(sel.sum()), coef[0], dtype=np.float64)
        for j in range(7):
            ts = ts + coef[1 + j] * x[j][sel]
        t[sel] = ts
    return t


def window_costs(models, decode_ctx, prefill, max_budget, t_cur, t_next):
    """(B_cur, B_sum, budgets, window costs): pred(b) + pred(B_sum - b) for every
    budget b in [|D|, min(B, B_cur)] (Eq. 16's objective)."""
    b_cur = time_to_budget(models, decode_ctx, prefill, max_budget, t_cur)
    b_sum = b_cur + time_to_budget(models, decode_ctx, prefill, max_budget, t_next)
    budgets = np.arange(len(decode_ctx), min(max_budget, b_cur) + 1, dtype=np.int64)
    costs = (preds_over_budgets(models, decode_ctx, prefill, budgets, max_budget)
             + preds_over_budgets(models, decode_ctx, prefill, b_sum - budgets, max_budget))
    return b_cur, b_sum, budgets, costs


def sliding_chunker(models, decode_ctx, prefill, max_budget, t_cur, t_next):
    """(budget, per-prefill chunks, predicted latency of this iteration): the
    budget minimising Eq. 16's window cost over every allowed budget, ties to the
    larger budget."""
    _, _, budgets, costs = window_costs(models, decode_ctx, prefill, max_budget, t_cur, t_next)
    best = int(budgets[costs == costs.min()].max())
    chunks, _, _ = form_batch(decode_ctx, prefill, best, max_budget)
    return best, chunks, pred_budget(models, decode_ctx, prefill, best, max_budget)
