"""SlidingChunker and TimeToBudget (Sec. 3.4, Alg. 1, Eq. 14-16).

The oracle (``oracle/chunker.py``: batch forming, TimeToBudget, and Eq. 16's
argmin over every budget) is pinned by batch forming worked by hand, by
TimeToBudget against a scan of every budget, by closed forms of the window
cost (a symmetric convex window splits B_sum evenly, with an exact tie at odd
B_sum that the larger budget wins; a flat window picks the largest budget) and
by the B_cur cap.  The library (``ssa_form_batch`` / ``ssa_time_to_budget`` /
``ssa_sliding_chunker``, an exact piecewise-quadratic search of its own) must
then reach the oracle's optimum: a window cost no worse than the exhaustive
minimum, the chunks its budget forms, and the same predicted latency bit for
bit, on random scheduler states with the same predictor loaded on both sides.
No GPU.
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


@pytest.mark.parametrize("seed", range(4))
def test_budget_sweep_matches_batch_forming(seed):
    # the oracle's pred over a whole budget range is the per-budget pred of the
    # hand-pinned batch forming, bit for bit
    rng = np.random.default_rng(50 + seed)
    dctx, pf, B = random_state(rng)
    budgets = np.arange(0, B + 40)
    got = orc.preds_over_budgets(MODELS, dctx, pf, budgets, B)
    ref = [orc.pred_budget(MODELS, dctx, pf, int(b), B) for b in budgets]
    assert got.tolist() == ref


def symmetric_state(b1, b2):
    """One prefill request with nothing cached, no decodes, and a predictor with
    only x2 = sum c^2 and x6 = sum c terms: pred(b) = w0 + w2 b^2 + w6 b for
    b >= 2, so the window cost pred(b) + pred(S - b) is symmetric about S / 2.
    T_cur and T_next are the predictions at b1 and b2, so B_cur = b1 and
    B_next = b2 (pred increases with b)."""
    models = {0: [1.0, 0.0, 1e-5, 0.0, 0.0, 0.0, 1e-3, 0.0]}
    pf, B = [(0, 6000)], 6000
    t_cur = orc.pred_budget(models, [], pf, b1, B)
    t_next = orc.pred_budget(models, [], pf, b2, B)
    return models, pf, B, t_cur, t_next


@pytest.mark.parametrize("b1,b2", [(1001, 500), (1000, 500), (3000, 777), (2500, 2499)])
def test_symmetric_window_splits_the_sum_evenly_ties_to_the_larger(b1, b2):
    models, pf, B, t_cur, t_next = symmetric_state(b1, b2)
    s = b1 + b2
    best, chunks, _ = orc.sliding_chunker(models, [], pf, B, t_cur, t_next)
    # even S: S / 2; odd S: (S - 1) / 2 and (S + 1) / 2 cost exactly the same
    # (the two terms swap), and the larger budget wins
    assert best == (s + 1) // 2
    assert chunks == [best]
    got = ssa.sliding_chunker(library_predictor(models), [], pf, B, t_cur, t_next)
    assert got[0] == best and got[1] == chunks


def test_flat_window_picks_the_largest_budget():
    # every non-empty batch is predicted at the intercept: the window cost is the
    # same for every budget (decodes keep both batches non-empty)
    models = {0: [25.0] + [0.0] * 7}
    dctx, pf, B = [100, 200, 300], [(0, 50), (7, 900)], 700
    best, chunks, _ = orc.sliding_chunker(models, dctx, pf, B, 30.0, 30.0)
    assert best == B and chunks == [50, 647]
    got = ssa.sliding_chunker(library_predictor(models), dctx, pf, B, 30.0, 30.0)
    assert got[0] == B and got[1] == chunks


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
def test_library_reaches_the_oracle_optimum(seed):
    rng = np.random.default_rng(300 + seed)
    dctx, pf, B = random_state(rng)
    p = library_predictor(MODELS)
    for t_cur, t_next in ((50.0, 80.0), (120.0, 60.0), (400.0, 400.0), (10.0, 10.0)):
        for b in (0, len(dctx), B // 2, B):
            assert ssa.form_batch(dctx, pf, b, B) == \
                tuple(list(v) if isinstance(v, list) else v for v in orc.form_batch(dctx, pf, b, B))
        assert ssa.time_to_budget(p, dctx, pf, B, t_cur) == \
            orc.time_to_budget(MODELS, dctx, pf, B, t_cur)
        _, _, budgets, costs = orc.window_costs(MODELS, dctx, pf, B, t_cur, t_next)
        ref = orc.sliding_chunker(MODELS, dctx, pf, B, t_cur, t_next)
        got = ssa.sliding_chunker(p, dctx, pf, B, t_cur, t_next)
        assert budgets[0] <= got[0] <= budgets[-1]
        lo = float(costs.min())
        mine = float(costs[got[0] - budgets[0]])
        assert mine <= lo + 1e-9 * max(1.0, abs(lo)), (got[0], ref[0], mine, lo)
        if np.sum(costs <= lo + 1e-9 * max(1.0, abs(lo))) == 1:
            assert got[0] == ref[0]
        assert got[1] == orc.form_batch(dctx, pf, got[0], B)[0]
        assert got[2] == orc.pred_budget(MODELS, dctx, pf, got[0], B)  # same fp64 sum, same order


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


@pytest.mark.parametrize("seed", range(12))
def test_plan_features_equal_batch_forming(seed):
    # the predictor is fitted on the planner's features of launched batches and
    # queried on batch forming's features: one rule for both, c = 0 and c = 1
    # prefill rows included
    rng = np.random.default_rng(900 + seed)
    dctx, pf, B = random_state(rng)
    pf = pf + [(int(rng.integers(0, 4000)), 1), (int(rng.integers(0, 4000)), 0)]
    rng.shuffle(pf)
    for b in (len(dctx), len(dctx) + 1, len(dctx) + 2, (len(dctx) + B) // 2, B):
        chunks, x, scene = ssa.form_batch(dctx, pf, b, B)
        q_len = [1] * len(dctx) + list(chunks)
        ctx = list(dctx) + [c for c, _ in pf]
        shape = ssa.make_shape(8, 2, 64, 1 << 20, 2048, 0.125)
        _, info = ssa.ssa_plan(shape, q_len, ctx)
        assert list(info.x) == list(x)
        assert info.scene == scene
