"""SlidingChunker and TimeToBudget (Sec. 3.4, Alg. 1, Eq. 14-16).

The oracle (``oracle/chunker.py``, Alg. 1 in the paper's order) is pinned by
batch forming worked by hand, by brute force (TimeToBudget against a scan of
every budget; the ternary search against the exact argmin of the window cost),
and by the B_cur cap.  The library (``ssa_form_batch`` / ``ssa_time_to_budget``
/ ``ssa_sliding_chunker``) must then take exactly the oracle's decisions: the
same budget and chunks, the same predicted latency bit for bit, on random
scheduler states with the same predictor loaded on both sides.  No GPU.
"""
import ctypes

import numpy as np
import pytest

from oracle import chunker as orc
from paper_2606_05933_amd import ssa

# a predictor in the shape of the fitted ones (us; per unit of each feature)
MODELS = {0: [60.0, 1.5e-5, -1e-5, 1.1e-3, 0.05, 1e-4, 2.5e-3, 5e-3],
          1: [36.0, 0.0, 0.0, 1.7e-4, 0.02, 1.7e-4, 0.0, 0.0],
          2: [67.0, 1.8e-5, -1.5e-5, 8e-4, 0.0, 0.0, 0.02, 0.01],
          3: [52.0, 1.3e-5, -3.5e-6, 1e-3, 0.05, 8e-4, 0.019, 0.003]}


def library_predictor(models):
    p = ssa.Predictor(min_scene_samples=1)
    for m, coef in models.items():
        for j, v in enumerate(coef):
            p.p.coef[m][j] = v
        p.p.fitted[m] = 1
    return p


def random_state(rng):
    nd = int(rng.integers(0, 128))
    dctx = [int(rng.integers(1, 16384)) for _ in range(nd)]
    prefill = [(int(rng.integers(0, 8192)), int(rng.integers(1, 4096)))
               for _ in range(int(rng.integers(0, 6)))]
    max_budget = nd + int(rng.integers(0, 8192))
    return dctx, prefill, max_budget


# ---------------------------------------------------------------- oracle pins

def test_batch_forming_worked_by_hand():
    dctx, pf = [100, 200], [(0, 50), (10, 5), (3, 100)]
    chunks, x, scene = orc.form_batch(dctx, pf, 60, 1000)
    assert chunks == [50, 5, 3]
    assert x == [50 * 50 + 5 * 15 + 3 * 6, 2500 + 25 + 9, 313, 2, 300, 58, 50]
    assert scene == orc.MIXED
    # two decodes and one token left: a one-token chunk is a decode row (Eq. 2)
    chunks, x, scene = orc.form_batch(dctx, pf, 3, 1000)
    assert chunks == [1, 0, 0] and x == [0, 0, 300, 3, 300, 0, 0] and scene == orc.PURE_DECODE
    # budgets below |D| are |D|; above B are B; no decode, no budget: empty
    assert orc.form_batch(dctx, pf, 0, 1000)[0] == [0, 0, 0]
    assert orc.form_batch(dctx, pf, 10 ** 6, 30)[0] == [28, 0, 0]
    assert orc.form_batch([], pf, 0, 30)[2] == 0
    assert orc.form_batch([], pf, 40, 40) == ([40, 0, 0], [1600.0, 1600.0, 0, 0, 0, 40.0, 40.0],
                                              orc.PURE_PREFILL)


@pytest.mark.parametrize("seed", range(6))
def test_time_to_budget_is_the_largest_budget_within_the_limit(seed):
    # non-negative weights: the prediction never decreases with the budget
    rng = np.random.default_rng(seed)
    models = {k: [abs(v) for v in c] for k, c in MODELS.items()}
    dctx, pf, B = random_state(rng)
    for t in np.linspace(0, 400, 17):
        got = orc.time_to_budget(models, dctx, pf, B, t)
        fits = [b for b in range(len(dctx), B + 1)
                if orc.pred_budget(models, dctx, pf, b, B) <= t]
        assert got == (max(fits) if fits else len(dctx))


@pytest.mark.parametrize("seed", range(8))
def test_ternary_search_lands_next_to_the_argmin_of_a_unimodal_window(seed):
    # only x6 (prefill tokens) and a convex x2 term: pred(b) + pred(S - b) is
    # convex in b, so Alg. 1's final interval holds the argmin
    rng = np.random.default_rng(100 + seed)
    models = {0: [10.0, 0, 2e-5, 0, 0, 0, 1e-2, 0]}
    dctx = [int(v) for v in rng.integers(1, 4096, size=int(rng.integers(1, 64)))]
    pf = [(0, int(rng.integers(500, 3000))) for _ in range(int(rng.integers(1, 4)))]
    B = len(dctx) + 4096
    b_cur, b_sum, costs = orc.window_costs(models, dctx, pf, B, 120.0, 160.0)
    best, chunks, t = orc.sliding_chunker(models, dctx, pf, B, 120.0, 160.0)
    lo_cost = min(costs.values())
    argmins = [b for b, c in costs.items() if c == lo_cost]
    # the pick is one of {l0, r0, m}, never worse than the ends, and m lies within
    # half of the final interval (at most 15) of the minimum
    assert costs[best] <= costs[len(dctx)] and costs[best] <= costs[min(B, b_cur)]
    assert best in (len(dctx), min(B, b_cur)) or min(abs(best - a) for a in argmins) <= 16
    assert chunks == orc.form_batch(dctx, pf, best, B)[0]
    assert t == orc.pred_budget(models, dctx, pf, best, B)


@pytest.mark.parametrize("seed", range(6))
def test_chunker_never_exceeds_the_current_window(seed):
    rng = np.random.default_rng(200 + seed)
    models = {k: [abs(v) for v in c] for k, c in MODELS.items()}
    dctx, pf, B = random_state(rng)
    for t_cur in (40.0, 90.0, 200.0):
        best, _, t = orc.sliding_chunker(models, dctx, pf, B, t_cur, 150.0)
        assert best <= orc.time_to_budget(models, dctx, pf, B, t_cur)
        if orc.pred_budget(models, dctx, pf, len(dctx), B) <= t_cur:
            assert t <= t_cur


# ----------------------------------------------------- library against oracle

@pytest.mark.parametrize("seed", range(40))
def test_library_takes_the_oracle_decisions(seed):
    rng = np.random.default_rng(300 + seed)
    dctx, pf, B = random_state(rng)
    p = library_predictor(MODELS)
    for t_cur, t_next in ((50.0, 80.0), (120.0, 60.0), (400.0, 400.0), (10.0, 10.0)):
        for b in (0, len(dctx), B // 2, B):
            assert ssa.form_batch(dctx, pf, b, B) == \
                tuple(list(v) if isinstance(v, list) else v for v in orc.form_batch(dctx, pf, b, B))
        assert ssa.time_to_budget(p, dctx, pf, B, t_cur) == \
            orc.time_to_budget(MODELS, dctx, pf, B, t_cur)
        got = ssa.sliding_chunker(p, dctx, pf, B, t_cur, t_next)
        ref = orc.sliding_chunker(MODELS, dctx, pf, B, t_cur, t_next)
        assert got[0] == ref[0] and got[1] == ref[1]
        assert got[2] == ref[2]  # same fp64 sum in the same order


def test_library_rejects_bad_arguments():
    L = ssa.LIB
    p = library_predictor(MODELS)
    d = (ctypes.c_int32 * 2)(5, 7)
    pf = (ssa.SsaPrefillRequest * 1)(ssa.SsaPrefillRequest(0, 10))
    ch = (ctypes.c_int32 * 1)()
    x = (ctypes.c_double * 7)()
    sc, b, t = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_double()
    assert L.ssa_form_batch(None, 2, pf, 1, 5, 10, ch, x, ctypes.byref(sc)) == -1
    assert L.ssa_form_batch(d, 2, pf, 1, 5, 10, None, x, ctypes.byref(sc)) == -1
    assert L.ssa_form_batch(d, -1, pf, 1, 5, 10, ch, x, ctypes.byref(sc)) == -13
    assert L.ssa_form_batch(d, 2, pf, 1, -5, 10, ch, x, ctypes.byref(sc)) == -13
    bad = (ssa.SsaPrefillRequest * 1)(ssa.SsaPrefillRequest(-1, 10))
    assert L.ssa_form_batch(d, 2, bad, 1, 5, 10, ch, x, ctypes.byref(sc)) == -13
    assert L.ssa_time_to_budget(None, d, 2, pf, 1, 10, 50.0, ctypes.byref(b)) == -1
    assert L.ssa_time_to_budget(ctypes.byref(p.p), d, 2, pf, 1, 1, 50.0, ctypes.byref(b)) == -13
    assert L.ssa_sliding_chunker(ctypes.byref(p.p), d, 2, pf, 1, 10, 50.0, 50.0, None, ch,
                                 ctypes.byref(t)) == -1
    unfitted = ssa.Predictor(1)
    assert L.ssa_sliding_chunker(ctypes.byref(unfitted.p), d, 2, pf, 1, 10, 50.0, 50.0,
                                 ctypes.byref(b), ch, ctypes.byref(t)) == -13
    assert L.ssa_sliding_chunker(ctypes.byref(p.p), d, 2, pf, 1, 10, 50.0, 50.0,
                                 ctypes.byref(b), ch, None) == 0  # t_pred is optional
