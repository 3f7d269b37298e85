"""CPU oracle of the batch latency predictor (SlidingServe Sec. 3.2).

TEST INFRASTRUCTURE ONLY: imported by ``tests/`` and by the benchmark's
predictor report, never by the library.  Plain numpy, float64; it imports
nothing from the library package.

What it computes, following Sec. 3.2:

* Eq. 2 sets: P = {c > 1}; D = {c <= 1} holds the requests with one new
  token.  A request with c = 0 has no new token this iteration and is not
  part of the batch that runs: it is in neither set, in no feature and decides
  no scene (the reading the planner and batch forming follow too).
* Eq. 3 scenes: pure decode (D only), pure prefill (P only), mixed; a batch
  with no new token has no scene.
* Tab. 1 features of a batch {(c_i, u_i)}: x1 = sum over P of c(u + c),
  x2 = sum over P of c^2, x3 = sum of u over the batch's requests (P and D),
  x4 = |D|, x5 = sum over D of u, x6 = sum over P of c, x7 = max over P of c
  (0 if P is empty).
* Eq. 5 per model: latency = b + sum_{j=1..7} w_j x_j.  (The printed sum runs
  over j = 0..7 with a separate intercept; read here as j = 1..7 plus b.)
* "Model training": a global model on all samples, and a scene's own model
  when that scene has at least ``min_scene_samples`` samples; prediction uses
  the scene's model when there is one, else the global model.
* The fit: least squares with the columns (1, x1..x7) scaled to unit
  sum of squares, columns that are zero on every sample left out, and a ridge
  of RIDGE on the scaled problem (it only decides how collinear columns share
  their weight; fitted values do not depend on that).  Solved by SVD least
  squares of the data matrix stacked on sqrt(RIDGE) * I.
* Tab. 5 metrics: MAE, RMSE, R^2 = 1 - SS_res / SS_tot.
"""
from __future__ import annotations

import numpy as np

RIDGE = 1e-10
SCENE_PURE_DECODE, SCENE_PURE_PREFILL, SCENE_MIXED = 1, 2, 3
SCENES = (SCENE_PURE_DECODE, SCENE_PURE_PREFILL, SCENE_MIXED)


def scene(q_len, ctx_len) -> int:
    """Eq. 3 scene of a batch (0 for an empty batch)."""
    c = np.asarray(q_len)
    n_p = int((c > 1).sum())
    n_d = int((c == 1).sum())
    if n_p + n_d == 0:
        return 0
    if n_p == 0:
        return SCENE_PURE_DECODE
    if n_d == 0:
        return SCENE_PURE_PREFILL
    return SCENE_MIXED


def features(q_len, ctx_len) -> np.ndarray:
    """Tab. 1 features x1..x7 of a batch, float64."""
    c = np.asarray(q_len, dtype=np.float64)
    u = np.asarray(ctx_len, dtype=np.float64)
    p = c > 1
    d = c == 1
    return np.array([
        float(np.sum(c[p] * (u[p] + c[p]))),
        float(np.sum(c[p] ** 2)),
        float(np.sum(u[p | d])),
        float(d.sum()),
        float(np.sum(u[d])),
        float(np.sum(c[p])),
        float(c[p].max()) if p.any() else 0.0,
    ])


def fit_linear(X, y) -> np.ndarray:
    """(b, w1..w7) of one model from samples X [n, 7], latencies y [n]."""
    X = np.asarray(X, dtype=np.float64).reshape(-1, 7)
    y = np.asarray(y, dtype=np.float64).reshape(-1)
    A = np.concatenate([np.ones((X.shape[0], 1)), X], axis=1)
    norm = np.sqrt(np.sum(A * A, axis=0))
    active = norm > 0
    As = A[:, active] / norm[active]
    k = As.shape[1]
    aug = np.concatenate([As, np.sqrt(RIDGE) * np.eye(k)], axis=0)
    rhs = np.concatenate([y, np.zeros(k)])
    sol, *_ = np.linalg.lstsq(aug, rhs, rcond=None)
    coef = np.zeros(8)
    coef[active] = sol / norm[active]
    return coef


def fit_models(X, scenes, y, min_scene_samples: int) -> dict:
    """{0: global coef, scene: coef for scenes with enough samples}."""
    X = np.asarray(X, dtype=np.float64).reshape(-1, 7)
    scenes = np.asarray(scenes)
    y = np.asarray(y, dtype=np.float64)
    models = {}
    if len(y):
        models[0] = fit_linear(X, y)
    for s in SCENES:
        m = scenes == s
        if int(m.sum()) >= min_scene_samples:
            models[s] = fit_linear(X[m], y[m])
    return models


def predict(models: dict, x, s: int) -> float:
    """The scene's model if fitted, else the global model."""
    coef = models.get(s, models.get(0))
    if coef is None:
        raise ValueError("no fitted model applies")
    return float(coef[0] + np.dot(coef[1:], np.asarray(x, dtype=np.float64)))


def metrics(y, yhat) -> dict:
    """Tab. 5: mean absolute error, root mean square error, R^2."""
    y = np.asarray(y, dtype=np.float64)
    yhat = np.asarray(yhat, dtype=np.float64)
    r = y - yhat
    ss_tot = float(np.sum((y - y.mean()) ** 2))
    return {"mae": float(np.mean(np.abs(r))), "rmse": float(np.sqrt(np.mean(r * r))),
            "r2": 1.0 - float(np.sum(r * r)) / ss_tot if ss_tot > 0 else float("nan")}
