// Batch latency predictor (SlidingServe Sec. 3.2: Eq. 3 scenes, Eq. 5 linear
// model per scene over the Tab. 1 features, global model plus scene experts,
// online incremental updates).  Host code; see include/ssa_predictor.h for the
// contract.

#include <cmath>
#include <cstring>

#include "../../include/ssa_predictor.h"

namespace {

constexpr int kF = SSA_PRED_FEATURES;  // features x1..x7
constexpr int kZ = kF + 2;             // z = (1, x1..x7, T)
constexpr int kN = kF + 1;             // unknowns (b, w1..w7)
// Ridge on the problem scaled to unit diagonal: far below any scale that
// matters for a fit, large enough that collinear features keep the system
// positive definite.
constexpr double kRidge = 1e-10;

static_assert(SSA_PRED_MOMENTS == kZ * (kZ + 1) / 2, "moment count");

// index of (i, j), i <= j, in the row-major upper triangle of a kZ x kZ matrix
constexpr int tri(int i, int j) { return i * kZ - i * (i - 1) / 2 + (j - i); }

bool valid_scene(int32_t s) {
  return s == SSA_SCENE_PURE_DECODE || s == SSA_SCENE_PURE_PREFILL || s == SSA_SCENE_MIXED;
}

// Least squares for one model from its moments: minimise sum (T - b - w.x)^2.
// The normal equations G c = g (G = sum x~ x~^T over x~ = (1, x), g = sum x~ T)
// are scaled to unit diagonal (features that are zero on every sample stay
// out), regularised by kRidge, and solved by Cholesky.  Returns false only if
// the model has no sample.
bool fit_model(const double* mom, int64_t n, double* coef) {
  for (int j = 0; j < kN; ++j) coef[j] = 0.0;
  if (n <= 0) return false;
  int idx[kN];
  int m = 0;
  double scale[kN];
  for (int j = 0; j < kN; ++j) {
    const double d = mom[tri(j, j)];
    if (d > 0.0 && std::isfinite(d)) {
      idx[m] = j;
      scale[m] = 1.0 / std::sqrt(d);
      ++m;
    }
  }
  double a[kN][kN], r[kN];
  for (int p = 0; p < m; ++p) {
    for (int q = 0; q < m; ++q) {
      const int i = idx[p] < idx[q] ? idx[p] : idx[q], j = idx[p] < idx[q] ? idx[q] : idx[p];
      a[p][q] = mom[tri(i, j)] * scale[p] * scale[q];
    }
    a[p][p] += kRidge;
    r[p] = mom[tri(idx[p], kZ - 1)] * scale[p];
  }
  // Cholesky a = L L^T in place (lower triangle)
  for (int p = 0; p < m; ++p) {
    for (int q = 0; q <= p; ++q) {
      double s = a[p][q];
      for (int k = 0; k < q; ++k) s -= a[p][k] * a[q][k];
      if (p == q) {
        a[p][p] = std::sqrt(s > 0.0 ? s : kRidge);
      } else {
        a[p][q] = s / a[q][q];
      }
    }
  }
  double y[kN];
  for (int p = 0; p < m; ++p) {  // L y = r
    double s = r[p];
    for (int k = 0; k < p; ++k) s -= a[p][k] * y[k];
    y[p] = s / a[p][p];
  }
  for (int p = m - 1; p >= 0; --p) {  // L^T c' = y
    double s = y[p];
    for (int k = p + 1; k < m; ++k) s -= a[k][p] * y[k];
    y[p] = s / a[p][p];
  }
  for (int p = 0; p < m; ++p) coef[idx[p]] = y[p] * scale[p];
  return true;
}

}  // namespace

extern "C" {

int ssa_predictor_init(ssa_predictor* p, int32_t min_scene_samples) {
  if (!p) return SSA_ERR_NULL;
  if (min_scene_samples < 1) return SSA_ERR_ARG;
  std::memset(p, 0, sizeof *p);
  p->min_scene_samples = min_scene_samples;
  return SSA_OK;
}

int ssa_predictor_add(ssa_predictor* p, const double* x, int32_t scene, double latency) {
  if (!p || !x) return SSA_ERR_NULL;
  if (!valid_scene(scene) || !std::isfinite(latency)) return SSA_ERR_ARG;
  double z[kZ];
  z[0] = 1.0;
  for (int j = 0; j < kF; ++j) {
    if (!std::isfinite(x[j])) return SSA_ERR_ARG;
    z[1 + j] = x[j];
  }
  z[kZ - 1] = latency;
  const int models[2] = {0, scene};
  for (int mi = 0; mi < 2; ++mi) {
    double* mom = p->moments[models[mi]];
    for (int i = 0; i < kZ; ++i)
      for (int j = i; j < kZ; ++j) mom[tri(i, j)] += z[i] * z[j];
    p->samples[models[mi]] += 1;
  }
  return SSA_OK;
}

int ssa_predictor_fit(ssa_predictor* p) {
  if (!p) return SSA_ERR_NULL;
  for (int m = 0; m < SSA_PRED_MODELS; ++m) {
    const int64_t need = m == 0 ? 1 : p->min_scene_samples;
    if (p->samples[m] >= need) {
      p->fitted[m] = fit_model(p->moments[m], p->samples[m], p->coef[m]) ? 1 : 0;
    } else {
      p->fitted[m] = 0;
      for (int j = 0; j < kN; ++j) p->coef[m][j] = 0.0;
    }
  }
  return SSA_OK;
}

int ssa_predictor_predict(const ssa_predictor* p, const double* x, int32_t scene,
                          double* latency) {
  if (!p || !x || !latency) return SSA_ERR_NULL;
  if (!valid_scene(scene)) return SSA_ERR_ARG;
  const int m = p->fitted[scene] ? scene : (p->fitted[0] ? 0 : -1);
  if (m < 0) return SSA_ERR_ARG;
  double t = p->coef[m][0];
  for (int j = 0; j < kF; ++j) t += p->coef[m][1 + j] * x[j];
  *latency = t;
  return SSA_OK;
}

}  // extern "C"
