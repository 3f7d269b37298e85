"""Batch latency predictor (Sec. 3.2: Eq. 3 scenes, Eq. 5, Tab. 1, Tab. 5 metrics).

The oracle (``oracle/predictor.py``) is pinned by what the mathematics fixes:
exact recovery of a planted linear model, agreement with plain least squares
on full-rank data, Tab. 1 features and Tab. 5 metrics worked by hand, and the
scene/global fallback rule.  The library's predictor (``ssa_predictor_*``,
normal equations solved by Cholesky) is then held to the oracle (SVD least
squares of the data matrix) on features of real plans.  No GPU.
"""
import ctypes

import numpy as np
import pytest

from oracle import predictor as orc
from paper_2606_05933_amd import ssa, workload

W_TRUE = {1: (40.0, [0, 0, 1e-4, 0.8, 0.011, 0, 0]),
          2: (25.0, [2e-6, 3e-6, 1e-4, 0, 0, 0.02, 0.01]),
          3: (60.0, [2.2e-6, 1e-6, 1.2e-4, 0.7, 0.01, 0.018, 0.005])}


def planted(x, s):
    b, w = W_TRUE[s]
    return b + float(np.dot(w, x))


def random_batch(rng, s):
    """(q_len, ctx_len) of a random batch of scene s."""
    nd = 0 if s == 2 else int(rng.integers(1, 200))
    npf = 0 if s == 1 else int(rng.integers(1, 5))
    c = [int(rng.integers(2, 2048)) for _ in range(npf)] + [1] * nd
    u = [int(rng.integers(0, 8192)) for _ in range(npf)] + \
        [int(rng.integers(16, 16384)) for _ in range(nd)]
    return c, u


def samples(n, seed, noise=0.0):
    rng = np.random.default_rng(seed)
    X, S, Y = [], [], []
    for k in range(n):
        s = 1 + k % 3
        c, u = random_batch(rng, s)
        x = orc.features(c, u)
        X.append(x)
        S.append(s)
        Y.append(planted(x, s) + noise * rng.standard_normal())
    return np.array(X), np.array(S), np.array(Y)


# ---------------------------------------------------------------- oracle pins

def test_features_and_scene_worked_by_hand():
    # P = {(5, 10), (3, 0)}, D = {(1, 7)}; the request (0, 4) has no new token
    # and is in neither set (the reading of Eq. 2 for c = 0)
    c, u = [5, 1, 3, 0], [10, 7, 0, 4]
    assert list(orc.features(c, u)) == [5 * 15 + 3 * 3, 25 + 9, 10 + 7 + 0, 1, 7, 8, 5]
    assert orc.scene(c, u) == orc.SCENE_MIXED
    assert orc.scene([1, 0], [3, 3]) == orc.SCENE_PURE_DECODE
    assert orc.scene([4, 2], [0, 9]) == orc.SCENE_PURE_PREFILL
    assert orc.scene([4, 0], [0, 9]) == orc.SCENE_PURE_PREFILL
    assert orc.scene([0, 0], [5, 9]) == 0
    assert list(orc.features([0, 0], [5, 9])) == [0] * 7
    assert orc.scene([], []) == 0


def test_features_match_the_planner():
    rng = np.random.default_rng(1)
    for s in (1, 2, 3):
        c, u = random_batch(rng, s)
        # requests with no new token this iteration, anywhere in the batch
        for _ in range(3):
            k = int(rng.integers(0, len(c) + 1))
            c.insert(k, 0)
            u.insert(k, int(rng.integers(0, 4096)))
        shape = ssa.make_shape(32, 8, 128, 1 << 20, max((a + b + 15) // 16 for a, b in zip(c, u)),
                               128 ** -0.5)
        _, info = ssa.ssa_plan(shape, c, u)
        assert list(info.x) == list(orc.features(c, u))
        assert info.scene == orc.scene(c, u)


def test_metrics_worked_by_hand():
    y = np.array([1.0, 2.0, 3.0, 4.0])
    assert orc.metrics(y, y) == {"mae": 0.0, "rmse": 0.0, "r2": 1.0}
    m = orc.metrics(y, y + 1.0)
    assert m["mae"] == 1.0 and m["rmse"] == 1.0 and abs(m["r2"] - (1 - 4 / 5)) < 1e-15
    m = orc.metrics(y, np.full(4, y.mean()))
    assert abs(m["r2"]) < 1e-15 and abs(m["rmse"] - np.sqrt(1.25)) < 1e-15


@pytest.mark.parametrize("s", [1, 2, 3])
def test_oracle_recovers_a_planted_model(s):
    X, S, Y = samples(300, seed=2)
    m = S == s
    coef = orc.fit_linear(X[m], Y[m])
    b, w = W_TRUE[s]
    pred = coef[0] + X[m] @ coef[1:]
    assert np.max(np.abs(pred - Y[m])) < 1e-6 * np.max(np.abs(Y[m]))
    assert orc.metrics(Y[m], pred)["r2"] > 1 - 1e-12
    if s == 3:  # every feature is present here: the weights themselves, up to what the
        # near-collinear features (x1, x2, x6, x7 all grow with c; x3 = x5 + the chunks'
        # u) let the tiny ridge move between them
        assert np.allclose(coef, [b] + w, rtol=1e-2, atol=1e-9)


def test_oracle_equals_plain_least_squares_on_full_rank_data():
    rng = np.random.default_rng(3)
    X = rng.uniform(0, 100, (60, 7))
    y = rng.normal(size=60) * 10 + X @ rng.normal(size=7)
    A = np.concatenate([np.ones((60, 1)), X], axis=1)
    ref, *_ = np.linalg.lstsq(A, y, rcond=None)
    assert np.allclose(orc.fit_linear(X, y), ref, rtol=1e-7, atol=1e-9)


def test_oracle_scene_model_needs_enough_samples():
    X, S, Y = samples(30, seed=4, noise=1.0)  # 10 per scene
    models = orc.fit_models(X, S, Y, min_scene_samples=11)
    assert set(models) == {0}
    models = orc.fit_models(X, S, Y, min_scene_samples=10)
    assert set(models) == {0, 1, 2, 3}
    only = orc.fit_models(X[:29], S[:29], Y[:29], min_scene_samples=10)  # scene 3 has 9
    assert set(only) == {0, 1, 2}
    g = orc.fit_linear(X[:29], Y[:29])
    assert orc.predict(only, X[2], 3) == pytest.approx(g[0] + X[2] @ g[1:], rel=1e-12)


# ----------------------------------------------------- library against oracle

def test_library_matches_the_oracle_on_plan_features():
    X, S, Y = samples(240, seed=5, noise=3.0)
    train = np.arange(len(Y)) % 4 != 0
    p = ssa.Predictor(min_scene_samples=20)
    for x, s, y in zip(X[train], S[train], Y[train]):
        p.add(x, s, y)
    p.fit()
    models = orc.fit_models(X[train], S[train], Y[train], min_scene_samples=20)
    for m in (0, 1, 2, 3):
        assert (p.coefficients(m) is not None) == (m in models)
    scale = np.max(np.abs(Y))
    got = np.array([p.predict(x, s) for x, s in zip(X, S)])
    ref = np.array([orc.predict(models, x, s) for x, s in zip(X, S)])
    assert np.max(np.abs(got - ref)) < 1e-7 * scale
    # the planted model is recovered up to the noise
    test = ~train
    assert orc.metrics(Y[test], got[test])["r2"] > 0.99


def test_library_weights_on_full_rank_data():
    rng = np.random.default_rng(6)
    X = rng.uniform(0, 1000, (80, 7))
    y = 3.0 + X @ np.array([1.5, -2.0, 0.25, 4.0, 0.0, 1e-3, 7.0])
    p = ssa.Predictor(min_scene_samples=1)
    for x, v in zip(X, y):
        p.add(x, 3, v)
    p.fit()
    assert np.allclose(p.coefficients(3), orc.fit_linear(X, y), rtol=1e-6, atol=1e-8)


def test_library_updates_online_and_copies_are_independent():
    X, S, Y = samples(90, seed=7, noise=2.0)
    once = ssa.Predictor(5)
    for x, s, y in zip(X, S, Y):
        once.add(x, s, y)
    once.fit()
    inc = ssa.Predictor(5)
    for x, s, y in zip(X[:40], S[:40], Y[:40]):
        inc.add(x, s, y)
    inc.fit()
    snapshot = inc.copy()
    for x, s, y in zip(X[40:], S[40:], Y[40:]):
        inc.add(x, s, y)
    inc.fit()
    for m in range(4):  # same moments in the same order: the same fit, bit for bit
        assert np.array_equal(once.coefficients(m), inc.coefficients(m))
    assert snapshot.p.samples[0] == 40 and inc.p.samples[0] == 90


def test_library_falls_back_to_the_global_model():
    X, S, Y = samples(12, seed=8, noise=1.0)  # 4 per scene
    p = ssa.Predictor(min_scene_samples=5)
    for x, s, y in zip(X, S, Y):
        p.add(x, s, y)
    p.fit()
    assert p.coefficients(0) is not None and all(p.coefficients(m) is None for m in (1, 2, 3))
    g = orc.fit_linear(X, Y)
    assert p.predict(X[0], 2) == pytest.approx(g[0] + X[0] @ g[1:], rel=1e-9)


def test_library_rejects_bad_arguments():
    L = ssa.LIB
    p = ssa.SsaPredictor()
    x = (ctypes.c_double * 7)(*([1.0] * 7))
    out = ctypes.c_double()
    assert L.ssa_predictor_init(None, 4) == -1
    assert L.ssa_predictor_init(ctypes.byref(p), 0) == -13
    assert L.ssa_predictor_init(ctypes.byref(p), 4) == 0
    assert L.ssa_predictor_add(ctypes.byref(p), None, 1, 1.0) == -1
    for bad_scene in (0, 4, -1):
        assert L.ssa_predictor_add(ctypes.byref(p), x, bad_scene, 1.0) == -13
    assert L.ssa_predictor_add(ctypes.byref(p), x, 1, float("nan")) == -13
    nan_x = (ctypes.c_double * 7)(*([1.0] * 6 + [float("inf")]))
    assert L.ssa_predictor_add(ctypes.byref(p), nan_x, 1, 1.0) == -13
    assert p.samples[0] == 0  # nothing written on an error
    assert L.ssa_predictor_predict(ctypes.byref(p), x, 1, ctypes.byref(out)) == -13  # no model
    assert L.ssa_predictor_add(ctypes.byref(p), x, 1, 5.0) == 0
    assert L.ssa_predictor_fit(ctypes.byref(p)) == 0
    assert L.ssa_predictor_predict(ctypes.byref(p), x, 1, ctypes.byref(out)) == 0
    assert out.value == pytest.approx(5.0)
    assert L.ssa_predictor_predict(ctypes.byref(p), x, 0, ctypes.byref(out)) == -13
    assert L.ssa_predictor_predict(ctypes.byref(p), x, 1, None) == -1
    assert L.ssa_predictor_fit(None) == -1
