"""Multi-Level Priority Sorter and BatchConstructor (Sec. 3.3, Eq. 6-13; Sec. 3.5,
Eq. 17-22, Alg. 2).

The oracle (``oracle/constructor.py``) is pinned by the priority keys worked by
hand, the value function worked by hand, the knapsack against every subset,
and Alg. 2 against an exhaustive search over every anchor and every subset.
The library (``ssa_priority_sort``, ``ssa_batch_constructor``) must then take
exactly the oracle's decisions on random scheduler states.  No GPU.
"""
import ctypes
import itertools

import numpy as np
import pytest

from oracle import chunker as och
from oracle import constructor as orc
from paper_2606_05933_amd import ssa

MODELS = {0: [60.0, 1.5e-5, -1e-5, 1.1e-3, 0.05, 1e-4, 2.5e-3, 5e-3],
          1: [36.0, 0.0, 0.0, 1.7e-4, 0.02, 1.7e-4, 0.0, 0.0],
          2: [67.0, 1.8e-5, -1.5e-5, 8e-4, 0.0, 0.0, 0.02, 0.01],
          3: [52.0, 1.3e-5, -3.5e-6, 1e-3, 0.05, 8e-4, 0.019, 0.003]}
EPS = 1e-3


def library_predictor(models):
    p = ssa.Predictor(min_scene_samples=1)
    for m, coef in models.items():
        for j, v in enumerate(coef):
            p.p.coef[m][j] = v
        p.p.fitted[m] = 1
    return p


def random_state(rng, n_max=8, slack=(-20.0, 300.0), nd_max=96):
    nd = int(rng.integers(0, nd_max))
    dctx = [int(rng.integers(1, 8192)) for _ in range(nd)]
    cands = [(int(rng.integers(0, 4096)), int(rng.integers(1, 1500)),
              float(np.round(rng.uniform(*slack), 3)), int(rng.random() < 0.2))
             for _ in range(int(rng.integers(1, n_max + 1)))]
    return dctx, cands, nd + int(rng.integers(64, 4096))


# states where most anchors are feasible and chosen sets hold several requests
ROOMY = {"slack": (60.0, 220.0), "nd_max": 24}


# ---------------------------------------------------------------- oracle pins

def test_priority_keys_worked_by_hand():
    # (cached, remaining, slack, safeguard); rho = 10 tokens per unit, alpha = 1
    cands = [(0, 100, 50.0, 0),   # u = 0.2: normal, r = 100
             (0, 10, 50.0, 0),    # u = 0.02: normal, r = 10
             (0, 500, 1.0, 0),    # u = 50: urgent
             (0, 300, 100.0, 1),  # safeguarded
             (0, 10, 80.0, 0),    # normal, r = 10: after the other r = 10 (input order)
             (0, 40, -5.0, 0)]    # late: s clamped to eps, u huge: urgent, r = 40
    assert orc.priority_sort(cands, 10.0, 1.0, EPS) == [3, 5, 2, 1, 4, 0]


def test_values_worked_by_hand():
    cands = [(0, 10, 1.0, 0), (0, 20, 2.0, 0), (0, 30, 3.0, 0)]
    # sum s = 6, sum r = 60: 1 / (1/6 + 1/6), 1 / (2/6 + 2/6), 1 / (3/6 + 3/6)
    assert orc.values(cands, [0, 1, 2], EPS) == pytest.approx([3.0, 1.5, 1.0], rel=1e-15)


@pytest.mark.parametrize("seed", range(20))
def test_knapsack_is_the_best_subset(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(0, 11))
    w = [int(v) for v in rng.integers(0, 40, size=n)]
    v = [float(x) for x in rng.uniform(0.1, 5.0, size=n)]
    cap = int(rng.integers(0, 120))
    chosen = orc.knapsack(w, v, cap)
    assert sum(w[i] for i in chosen) <= cap
    best = max(sum(v[i] for i in s) for k in range(n + 1)
               for s in itertools.combinations(range(n), k) if sum(w[i] for i in s) <= cap)
    assert sum(v[i] for i in chosen) == pytest.approx(best, rel=1e-12)


def exhaustive(models, dctx, cands, B):
    """Alg. 2 as a definition: for every feasible risky anchor, the subset of
    the requests with no less slack (anchor included) of most total value
    within the anchor's capacity, compared by (|Y|, sum v, sum r)."""
    pf = [(c[0], c[1]) for c in cands]
    t_full = och.pred_budget(models, dctx, pf, B, B)
    risky = [k for k, c in enumerate(cands) if c[2] < t_full]
    if not risky:
        return orc.NO_RISK, None
    order = sorted(range(len(cands)), key=lambda k: (cands[k][2], cands[k][1]))
    best = None
    for a in [k for k in order if k in risky]:
        cap = min(B, och.time_to_budget(models, dctx, pf, B, cands[a][2])) - len(dctx)
        if cap <= 0 or cands[a][1] > cap:
            continue
        s_a = [j for j in order if cands[j][2] >= cands[a][2]]
        vals = dict(zip(s_a, orc.values(cands, s_a, EPS)))
        others = [j for j in s_a if j != a]
        top = None
        for k in range(len(others) + 1):
            for sub in itertools.combinations(others, k):
                if sum(cands[j][1] for j in sub) <= cap - cands[a][1]:
                    val = sum(vals[j] for j in sub)
                    if top is None or val > top[0] + 1e-12:
                        top = (val, set(sub))
        y = top[1] | {a}
        key = (len(y), sum(vals[j] for j in y), sum(cands[j][1] for j in y))
        if best is None or key[0] > best[0][0] or (key[0] == best[0][0] and
                                                   key[1] > best[0][1] + 1e-12):
            best = (key, y)
    if best is None:
        return orc.NO_ANCHOR, None
    return orc.BATCH, best[1]


@pytest.mark.parametrize("seed", range(60))
def test_constructor_is_the_exhaustive_best(seed):
    rng = np.random.default_rng(1000 + seed)
    dctx, cands, B = random_state(rng, n_max=7, **(ROOMY if seed % 2 else {}))
    outcome, budget, take, t_full = orc.batch_constructor(MODELS, dctx, cands, B, EPS)
    ref_outcome, ref_set = exhaustive(MODELS, dctx, cands, B)
    assert outcome == ref_outcome
    if outcome == orc.BATCH:
        assert {k for k, t in enumerate(take) if t} == ref_set
        assert budget == len(dctx) + sum(cands[k][1] for k in ref_set)
        assert all(t in (0, cands[k][1]) for k, t in enumerate(take))


def test_constructor_outcomes():
    dctx = [1000] * 20
    calm = [(0, 200, 1e6, 0), (0, 300, 1e6, 0)]
    assert orc.batch_constructor(MODELS, dctx, calm, 2000, EPS)[0] == orc.NO_RISK
    hopeless = [(0, 200, 1.0, 0), (0, 300, 2.0, 0)]  # slack below even the decodes' time
    assert orc.batch_constructor(MODELS, dctx, hopeless, 2000, EPS)[0] == orc.NO_ANCHOR


# ----------------------------------------------------- library against oracle

@pytest.mark.parametrize("seed", range(80))
def test_library_takes_the_oracle_decisions(seed):
    rng = np.random.default_rng(2000 + seed)
    dctx, cands, B = random_state(rng, n_max=12, **(ROOMY if seed % 2 else {}))
    for rho, alpha in ((5.0, 1.0), (50.0, 0.5), (1.0, 4.0)):
        assert ssa.priority_sort(cands, rho, alpha, EPS) == orc.priority_sort(cands, rho, alpha, EPS)
    order = orc.priority_sort(cands, 20.0, 1.0, EPS)
    sorted_cands = [cands[k] for k in order]
    p = library_predictor(MODELS)
    got = ssa.batch_constructor(p, dctx, sorted_cands, B, EPS)
    ref = orc.batch_constructor(MODELS, dctx, sorted_cands, B, EPS)
    assert got == ref


def test_library_rejects_bad_arguments():
    L = ssa.LIB
    p = library_predictor(MODELS)
    c = (ssa.SsaCandidate * 1)(ssa.SsaCandidate(0, 10, 5.0, 0, 0))
    order = (ctypes.c_int32 * 1)()
    d = (ctypes.c_int32 * 1)(100)
    oc, b, tf = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_double()
    take = (ctypes.c_int32 * 1)()
    assert L.ssa_priority_sort(None, 1, 1.0, 1.0, 1e-3, order) == -1
    assert L.ssa_priority_sort(c, 1, 0.0, 1.0, 1e-3, order) == -13
    assert L.ssa_priority_sort(c, 1, 1.0, 1.0, 0.0, order) == -13
    nan = (ssa.SsaCandidate * 1)(ssa.SsaCandidate(0, 10, float("nan"), 0, 0))
    assert L.ssa_priority_sort(nan, 1, 1.0, 1.0, 1e-3, order) == -13
    args = (ctypes.byref(oc), ctypes.byref(b), take, ctypes.byref(tf))
    assert L.ssa_batch_constructor(None, d, 1, c, 1, 100, 1e-3, *args) == -1
    assert L.ssa_batch_constructor(ctypes.byref(p.p), d, 1, c, 1, 100, 0.0, *args) == -13
    assert L.ssa_batch_constructor(ctypes.byref(p.p), d, 1, c, 1, 0, 1e-3, *args) == -13
    assert L.ssa_batch_constructor(ctypes.byref(p.p), d, 1, c, 1, 1 << 21, 1e-3, *args) == -13
    assert L.ssa_batch_constructor(ctypes.byref(p.p), d, 1, c, 1, 100, 1e-3,
                                   None, ctypes.byref(b), take, None) == -1
