"""CPU oracle of SlidingChunker and TimeToBudget (SlidingServe Sec. 3.4, Alg. 1).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, never by the library.  Plain
Python integers and floats; it imports nothing from the library package.

It follows Alg. 1 in the paper's order:

1. B_cur = TimeToBudget(T_cur), B_next = TimeToBudget(T_next) (binary search,
   "approximated using binary search", Sec. 3.4);
2. B_sum = B_cur + B_next;
3. l = |D|, r = B (here capped by B_cur: the printed algorithm never bounds b by
   B_cur, which could pick a budget that breaks this iteration's bound);
4. discrete ternary search on pred(b) + pred(B_sum - b) (Eq. 16) while r - l > 30;
5. the candidates {l0, r0, floor((l + r) / 2)}: the least window cost, ties to the
   larger budget.

Batch forming (BatchForwarder): decodes take one token each; the rest of the
budget goes to the sorted prefill requests in order, min(remaining, left) each.
Budgets are clamped to [|D|, B].  The formed batch's features are Tab. 1 with
Eq. 2's split (a request given one token is a decode row; one given none is not
in the batch), and an empty batch takes no time.

The predictor is a dict {0: global, scene: model} of (b, w1..w7), evaluated as
b + w1 x1 + ... + w7 x7 in that order (Eq. 5), the scene's model first.
"""
from __future__ import annotations

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


def sliding_chunker(models, decode_ctx, prefill, max_budget, t_cur, t_next):
    """Alg. 1: (budget, chunks, predicted latency of this iteration)."""
    def pred(b):
        return pred_budget(models, decode_ctx, prefill, b, max_budget)

    b_cur = time_to_budget(models, decode_ctx, prefill, max_budget, t_cur)
    b_next = time_to_budget(models, decode_ctx, prefill, max_budget, t_next)
    b_sum = b_cur + b_next
    l, r = len(decode_ctx), min(max_budget, b_cur)
    l0, r0 = l, r
    while r - l > 30:
        m1 = l + (r - l) // 3
        m2 = r - (r - l) // 3
        if pred(m1) + pred(b_sum - m1) <= pred(m2) + pred(b_sum - m2):
            r = m2 - 1
        else:
            l = m1 + 1
    best, best_cost = None, None
    for b in (l0, r0, l + (r - l) // 2):
        c = pred(b) + pred(b_sum - b)
        if best is None or c < best_cost or (c == best_cost and b > best):
            best, best_cost = b, c
    chunks, _, _ = form_batch(decode_ctx, prefill, best, max_budget)
    return best, chunks, pred(best)


def window_costs(models, decode_ctx, prefill, max_budget, t_cur, t_next):
    """Brute force: (B_cur, B_sum, {b: pred(b) + pred(B_sum - b)}) over every
    budget Alg. 1 may pick."""
    b_cur = time_to_budget(models, decode_ctx, prefill, max_budget, t_cur)
    b_sum = b_cur + time_to_budget(models, decode_ctx, prefill, max_budget, t_next)
    costs = {b: pred_budget(models, decode_ctx, prefill, b, max_budget)
             + pred_budget(models, decode_ctx, prefill, b_sum - b, max_budget)
             for b in range(len(decode_ctx), min(max_budget, b_cur) + 1)}
    return b_cur, b_sum, costs
