/*
 * ssa_predictor.h -- batch latency predictor of a serving iteration
 * (SlidingServe Sec. 3.2, Eq. 3 scenes, Eq. 5 model, Tab. 1 features).
 *
 * Host-only C ABI, compiled into libssa.so beside the attention path.  The
 * predictor estimates the latency of one iteration from the seven batch
 * features x1..x7 of Tab. 1 (ssa_plan fills them into ssa_plan_info.x, and the
 * scene into ssa_plan_info.scene):
 *
 *     T_hat = b(m) + sum_{j=1..7} w_j(m) * x_j          (Eq. 5, read as j = 1..7
 *                                                        plus the intercept b)
 *
 * with one linear model per scene m (pure decode, pure prefill, mixed; Eq. 3)
 * and one global model over all samples.  A scene's own ("expert") model is
 * fitted once that scene has at least min_scene_samples samples; prediction
 * uses it when fitted and falls back to the global model otherwise (Sec. 3.2,
 * "Model training").
 *
 * Samples are accumulated as second moments (sum of z z^T with
 * z = (1, x1, .., x7, T), fp64), so adding a sample is O(1) and a model can be
 * refitted at any time from everything seen so far: the paper's online
 * incremental update.  The struct is plain data owned by the caller; a caller
 * that refits in the background fits a copy and swaps it in (the paper's hot
 * switch).  The library allocates nothing and keeps no state.
 *
 * The fit is least squares on the features scaled to unit second moment,
 * with a ridge of 1e-10 on the scaled problem: features that are zero on
 * every sample of a model drop out, and collinear ones (x6 = x7 when a batch
 * has one chunk, x4 constant, ...) get the minimum-norm split of their weight.
 * Fitted values do not depend on that split.
 *
 * All calls return 0 or a negative SSA_ERR_* code (ssa.h), validate before
 * writing, and write nothing on an error.
 */
#ifndef SSA_PREDICTOR_H
#define SSA_PREDICTOR_H

#include <stdint.h>

#include "ssa.h"

#ifdef __cplusplus
extern "C" {
#endif

#define SSA_PRED_FEATURES 7 /* x1..x7 */
#define SSA_PRED_MODELS 4   /* 0: global; 1, 2, 3: SSA_SCENE_PURE_DECODE, _PURE_PREFILL, _MIXED */
#define SSA_PRED_MOMENTS 45 /* upper triangle of the 9 x 9 matrix sum z z^T */

typedef struct ssa_predictor {
  int64_t samples[SSA_PRED_MODELS];                 /* samples seen by each model */
  double moments[SSA_PRED_MODELS][SSA_PRED_MOMENTS]; /* row-major upper triangle */
  double coef[SSA_PRED_MODELS][1 + SSA_PRED_FEATURES]; /* b, w1..w7 where fitted */
  int32_t fitted[SSA_PRED_MODELS];                  /* 1 once ssa_predictor_fit fitted it */
  int32_t min_scene_samples;                        /* samples a scene model needs */
  int32_t reserved;
} ssa_predictor;

/*
 * Empty predictor.  min_scene_samples >= 1: the samples a scene needs for its
 * own model.  Errors: SSA_ERR_NULL (p), SSA_ERR_ARG (min_scene_samples < 1).
 */
int ssa_predictor_init(ssa_predictor* p, int32_t min_scene_samples);

/*
 * One measured iteration: its features x[0..6] = x1..x7, its scene
 * (SSA_SCENE_PURE_DECODE, _PURE_PREFILL or _MIXED) and its latency (any time
 * unit; predictions come back in the same unit).  Counts in the global model
 * and in the scene's.  Errors: SSA_ERR_NULL (p, x), SSA_ERR_ARG (another
 * scene, or a non-finite feature or latency).
 */
int ssa_predictor_add(ssa_predictor* p, const double* x, int32_t scene, double latency);

/*
 * Fit the global model (if it has a sample) and every scene model with at
 * least min_scene_samples samples, from all samples added so far; models with
 * too few samples are marked not fitted.  Errors: SSA_ERR_NULL.
 */
int ssa_predictor_fit(ssa_predictor* p);

/*
 * Predicted latency of a batch with features x[0..6] in the given scene: the
 * scene's model if fitted, else the global model.  Errors: SSA_ERR_NULL
 * (p, x, latency), SSA_ERR_ARG (scene not 1..3, or no fitted model applies).
 */
int ssa_predictor_predict(const ssa_predictor* p, const double* x, int32_t scene,
                          double* latency);

#ifdef __cplusplus
}
#endif

#endif /* SSA_PREDICTOR_H */
