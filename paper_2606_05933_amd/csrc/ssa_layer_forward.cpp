// One decoder layer as a sequence of the library's launches
// (include/ssa_layer.h): host code only.  All sizes, pointers, positions and
// the workspace are checked before the first launch.
#include <stddef.h>
#include <stdint.h>

#include <algorithm>
#include <cmath>

#include "../../include/ssa_layer.h"
#include "ssa_plan_format.h"

namespace ssa {
int check_plan(const ssa_shape* s, const void* plan_host, const PlanHeader** out);
}

namespace {
using namespace ssa;

size_t align256(size_t b) { return (b + 255) / 256 * 256; }

// Byte offsets of the regions of the layer workspace.  The attention and
// linear workspaces (whose counters must stay zero at rest) come first.
struct LayerWs {
  size_t attn, gemm, xn, qkv, q, a, h, act, total;
  size_t attn_bytes, gemm_bytes;
};

int layer_ws(const ssa_shape* shape, const void* plan_host, const ssa_layer_weights* w,
             const PlanHeader** hdr, LayerWs* l) {
  if (!shape || !plan_host || !w || !hdr || !l) return SSA_ERR_NULL;
  const PlanHeader* h = nullptr;
  int rc = check_plan(shape, plan_host, &h);
  if (rc) return rc;
  const int64_t t = h->num_tokens;
  const int64_t qd = (int64_t)h->hq * h->head_dim;
  const int64_t nqkv = (int64_t)(h->hq + 2 * h->hkv) * h->head_dim;
  if (w->hidden <= 0 || w->hidden % 128 || w->hidden > 8192 || w->inter <= 0 || w->inter % 64 ||
      nqkv % 128 || !(w->eps >= 0.f) || w->max_position < 0)
    return SSA_ERR_ARG;
  size_t g = 0, b = 0;
  const int32_t m = (int32_t)t;
  if ((rc = ssa_linear_workspace_size(m, (int32_t)nqkv, w->hidden, &b))) return rc;
  g = std::max(g, b);
  if ((rc = ssa_linear_workspace_size(m, w->hidden, (int32_t)qd, &b))) return rc;
  g = std::max(g, b);
  if ((rc = ssa_linear_workspace_size(m, 2 * w->inter, w->hidden, &b))) return rc;
  g = std::max(g, b);
  if ((rc = ssa_linear_workspace_size(m, w->hidden, w->inter, &b))) return rc;
  g = std::max(g, b);
  l->attn_bytes = (size_t)h->ws_bytes;
  l->gemm_bytes = g;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += align256(bytes);
    return o;
  };
  l->attn = take(l->attn_bytes);
  l->gemm = take(l->gemm_bytes);
  l->xn = take((size_t)t * w->hidden * 2);
  l->qkv = take((size_t)t * nqkv * 2);
  l->q = take((size_t)t * qd * 2);
  l->a = take((size_t)t * qd * 2);
  l->h = take((size_t)t * w->hidden * 2);
  l->act = take((size_t)t * w->inter * 2);
  l->total = off;
  *hdr = h;
  return SSA_OK;
}

}  // namespace

extern "C" {

int ssa_rope_table(int32_t max_position, int32_t d, double base, float* out) {
  if (!out) return SSA_ERR_NULL;
  if (max_position < 1 || d < 2 || d % 2 || !std::isfinite(base) || !(base > 1.0)) return SSA_ERR_ARG;
  const int half = d / 2;
  for (int i = 0; i < half; ++i) {
    const double t = std::pow(base, -2.0 * i / d);
    for (int64_t p = 0; p < max_position; ++p) {
      const double a = (double)p * t;
      out[p * d + i] = (float)std::cos(a);
      out[p * d + half + i] = (float)std::sin(a);
    }
  }
  return SSA_OK;
}

int ssa_layer_workspace_size(const ssa_shape* shape, const void* plan_host,
                             const ssa_layer_weights* w, size_t* ws_bytes) {
  if (!ws_bytes) return SSA_ERR_NULL;
  const PlanHeader* h = nullptr;
  LayerWs l;
  const int rc = layer_ws(shape, plan_host, w, &h, &l);
  if (rc) return rc;
  *ws_bytes = l.total;
  return SSA_OK;
}

int ssa_layer_forward(const ssa_shape* shape, const void* plan_host, const void* plan_dev,
                      const ssa_layer_weights* w, const uint16_t* x, uint16_t* out,
                      uint16_t* k_cache, uint16_t* v_cache, const int32_t* block_table,
                      void* workspace, size_t ws_bytes, void* stream) {
  const PlanHeader* h = nullptr;
  LayerWs l;
  int rc = layer_ws(shape, plan_host, w, &h, &l);
  if (rc) return rc;
  if (!plan_dev) return SSA_ERR_NULL;
  const ReqEntry* reqs =
      reinterpret_cast<const ReqEntry*>(static_cast<const uint8_t*>(plan_host) + h->off_reqs);
  for (int32_t i = 0; i < h->num_reqs; ++i)
    if (reqs[i].q_len > 0 && (int64_t)reqs[i].ctx_len + reqs[i].q_len > w->max_position)
      return SSA_ERR_ARG;
  const int32_t t = h->num_tokens;
  if (t == 0) return SSA_OK;
  if (!x || !out || !k_cache || !v_cache || !block_table || !w->attn_norm || !w->w_qkv ||
      !w->w_o || !w->mlp_norm || !w->w_gate_up || !w->w_down || !w->cos_sin)
    return SSA_ERR_NULL;
  if (!workspace || ws_bytes < l.total) return SSA_ERR_WORKSPACE;
  char* ws = static_cast<char*>(workspace);
  auto at = [&](size_t off) { return reinterpret_cast<uint16_t*>(ws + off); };
  uint16_t *xn = at(l.xn), *qkv = at(l.qkv), *q = at(l.q), *a = at(l.a), *hb = at(l.h),
           *act = at(l.act);
  void* gws = ws + l.gemm;
  const int32_t hid = w->hidden, qd = h->hq * h->head_dim;
  const int32_t nqkv = (h->hq + 2 * h->hkv) * h->head_dim;

  if ((rc = ssa_rms_norm(t, hid, x, w->attn_norm, w->eps, xn, stream))) return rc;
  if ((rc = ssa_linear(t, nqkv, hid, SSA_EPILOGUE_NONE, xn, w->w_qkv, nullptr, qkv, gws,
                       l.gemm_bytes, stream)))
    return rc;
  if ((rc = ssa_rope_append(shape, plan_host, plan_dev, qkv, w->cos_sin, w->max_position, q,
                            k_cache, v_cache, block_table, stream)))
    return rc;
  if ((rc = ssa_mixed_attention(shape, plan_host, plan_dev, q, k_cache, v_cache, block_table, a,
                                ws + l.attn, l.attn_bytes, stream)))
    return rc;
  if ((rc = ssa_linear(t, hid, qd, SSA_EPILOGUE_RESIDUAL, a, w->w_o, x, hb, gws, l.gemm_bytes,
                       stream)))
    return rc;
  if ((rc = ssa_rms_norm(t, hid, hb, w->mlp_norm, w->eps, xn, stream))) return rc;
  if ((rc = ssa_linear(t, 2 * w->inter, hid, SSA_EPILOGUE_SWIGLU, xn, w->w_gate_up, nullptr, act,
                       gws, l.gemm_bytes, stream)))
    return rc;
  return ssa_linear(t, hid, w->inter, SSA_EPILOGUE_RESIDUAL, act, w->w_down, hb, out, gws,
                    l.gemm_bytes, stream);
}

}  // extern "C"
