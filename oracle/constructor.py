"""CPU oracle of the Multi-Level Priority Sorter and the BatchConstructor
(SlidingServe Sec. 3.3, Eq. 6-13; Sec. 3.5, Eq. 17-22, Alg. 2).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, never by the library.  Plain
Python; batch forming, prediction and TimeToBudget come from
``oracle/chunker.py``.

Priority sort: u_i = r_i / (rho * max(s_i, eps)) (Eq. 10), e_i = [u_i > alpha]
(Eq. 11), ascending on (1 - g_i, 1 - e_i, r_i) (Eq. 12-13), ties in input order.

Alg. 2, in the paper's order, on candidates (cached, remaining, slack, safeguard)
already in priority order:
  T_full = pred(the batch the full budget forms); risky = {j : s_j < T_full};
  none -> "no risk".  C = candidates by increasing (s, r) (read for the printed
  undefined "sort C"); for each risky anchor a in C order: B_a = TimeToBudget(s_a),
  C_a = min(B, B_a) - |D|, skip if C_a <= 0 or r_a > C_a; S_a = {j in C : s_j >= s_a};
  v_j = 1 / (s'_j / sum s' + r_j / sum r) over S_a with s' = max(s, eps) (Eq. 18);
  Y = 0/1 knapsack over S_a \\ {a} within C_a - r_a (Eq. 19), plus a (Eq. 20);
  keep Y if (|Y|, sum v, sum r) beats the best so far (Eq. 21, strict).  No
  feasible anchor -> "no anchor".  Otherwise budget |D| + sum r, every chosen
  request given all its remaining tokens (Eq. 22).

Parity unpinned: the third key of Eq. 21 (sum r).  Two anchors with equal slack
share S_a, Eq. 18's values and their capacity, so they reach the same set; anchors
with different slack normalise Eq. 18 over different sets, so an exact tie of
(|Y|, sum v) between different sets needs a numeric coincidence.  No pin state
with such a tie is known (an exact-arithmetic search of 300,000 small states
found none), so no test fails when this key is dropped.
"""
from __future__ import annotations

from oracle import chunker as ch

NO_RISK, NO_ANCHOR, BATCH = 0, 1, 2


def priority_sort(cands, throughput, alpha, eps):
    def key(k):
        cached, r, s, g = cands[k]
        u = r / (throughput * max(s, eps))
        return (0 if g else 1, 0 if u > alpha else 1, r)
    return sorted(range(len(cands)), key=key)


def knapsack(weights, values, cap):
    """Most total value within cap; items in order, a later item replacing an
    earlier choice only when strictly better.  Chosen item positions."""
    best = [0.0] * (cap + 1)
    keep = [[False] * (cap + 1) for _ in weights]
    for i, (w, v) in enumerate(zip(weights, values)):
        for c in range(cap, w - 1, -1):
            cand = best[c - w] + v
            if cand > best[c]:
                best[c] = cand
                keep[i][c] = True
    chosen, c = [], cap
    for i in range(len(weights) - 1, -1, -1):
        if keep[i][c]:
            chosen.append(i)
            c -= weights[i]
    return sorted(chosen)


def values(cands, s_a, eps):
    sum_s = 0.0
    sum_r = 0
    for j in s_a:
        sum_s += max(cands[j][2], eps)
        sum_r += cands[j][1]
    out = []
    for j in s_a:
        rr = cands[j][1] / sum_r if sum_r > 0 else 0.0
        out.append(1.0 / (max(cands[j][2], eps) / sum_s + rr))
    return out


def batch_constructor(models, decode_ctx, cands, max_budget, eps):
    """(outcome, budget, per-candidate tokens, T_full)."""
    pf = [(c[0], c[1]) for c in cands]
    t_full = ch.pred_budget(models, decode_ctx, pf, max_budget, max_budget)
    if not any(c[2] < t_full for c in cands):
        return NO_RISK, None, None, t_full
    order = sorted(range(len(cands)), key=lambda k: (cands[k][2], cands[k][1]))
    nd = len(decode_ctx)
    best = None  # (n, sum v, sum r, set)
    for a in order:
        s_anchor, r_anchor = cands[a][2], cands[a][1]
        if not s_anchor < t_full:
            continue
        b_a = ch.time_to_budget(models, decode_ctx, pf, max_budget, s_anchor)
        cap_a = min(max_budget, b_a) - nd
        if cap_a <= 0 or r_anchor > cap_a:
            continue
        s_a = [j for j in order if cands[j][2] >= s_anchor]
        vals = values(cands, s_a, eps)
        items = [k for k, j in enumerate(s_a) if j != a]
        chosen = knapsack([cands[s_a[k]][1] for k in items], [vals[k] for k in items],
                          cap_a - r_anchor)
        in_y = {items[p] for p in chosen} | {s_a.index(a)}
        yn, yv, yr = 0, 0.0, 0
        for k, j in enumerate(s_a):
            if k in in_y:
                yn += 1
                yv += vals[k]
                yr += cands[j][1]
        if best is None or (yn, yv, yr) > best[:3]:
            best = (yn, yv, yr, {s_a[k] for k in in_y})
    if best is None:
        return NO_ANCHOR, None, None, t_full
    take = [cands[k][1] if k in best[3] else 0 for k in range(len(cands))]
    return BATCH, nd + best[2], take, t_full
