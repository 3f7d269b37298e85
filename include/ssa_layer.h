/*
 * ssa_layer.h -- the GPU steps around attention in one transformer layer of a
 * serving iteration (Llama-3-8B: RMSNorm, QKV projection, rotary position
 * embedding, attention over the paged cache, O projection, RMSNorm, SwiGLU
 * MLP).  They measure what the linear layers add to an iteration's latency,
 * the cost the paper's features x6 and x7 stand for (Tab. 1).
 *
 * Same conventions as ssa.h: 0 or a negative SSA_ERR_* code, validation before
 * any HIP call, nothing written on an error, no allocation; bf16 as uint16_t
 * bit patterns; arithmetic in fp32 with round-to-nearest-even to bf16.
 */
#ifndef SSA_LAYER_H
#define SSA_LAYER_H

#include <stddef.h>
#include <stdint.h>

#include "ssa.h"

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Rotary position embedding of the new tokens' queries and keys, and kv_append
 * of the rotated keys and the values, in one launch (one workgroup per append
 * segment of the plan).
 *   qkv      [T, (Hq + 2 Hkv) D] bf16: the QKV projection of the T new tokens,
 *            per row the Hq query heads, then the Hkv key heads, then the Hkv
 *            value heads, D each (rows in plan order, as q in ssa.h)
 *   cos_sin  [max_position, D] fp32: row p holds cos(p t_i) in columns i < D/2
 *            and sin(p t_i) in columns D/2 + i, t_i = base^(-2i/D)
 *   q_out    [T, Hq, D] bf16: the rotated queries (the q of ssa_mixed_attention)
 *   k_cache, v_cache, block_table: as ssa_kv_append; the rotated key and the
 *            value of the token at position u_i + j go to that position's slot
 * Rotation (the "rotate half" pairing): for dims i < D/2 of a head,
 *   out[i] = x[i] cos - x[i + D/2] sin,  out[i + D/2] = x[i + D/2] cos + x[i] sin,
 * with (cos, sin) the row of the token's position.  Values are copied bit for
 * bit.  Every pool byte outside the new slots is left as it is.
 * Errors: those of ssa_kv_append; SSA_ERR_NULL (qkv, cos_sin, q_out);
 * SSA_ERR_ARG (a new token's position u_i + j >= max_position).
 */
int ssa_rope_append(const ssa_shape* shape, const void* plan_host, const void* plan_dev,
                    const uint16_t* qkv, const float* cos_sin, int32_t max_position,
                    uint16_t* q_out, uint16_t* k_cache, uint16_t* v_cache,
                    const int32_t* block_table, void* stream);

/*
 * The rotary table of ssa_rope_append, on the host: out [max_position, d] fp32
 * (caller's buffer), row p = cos(p t_i) for i < d/2, then sin(p t_i), with
 * t_i = base^(-2i/d); angles and functions in fp64, each entry rounded once to
 * fp32.  Errors: SSA_ERR_NULL (out); SSA_ERR_ARG (max_position < 1, d < 2 or
 * odd, base <= 1 or not finite).  Allocates nothing.
 */
int ssa_rope_table(int32_t max_position, int32_t d, double base, float* out);

/* Epilogues of ssa_linear. */
enum {
  SSA_EPILOGUE_NONE = 0,     /* out = x W^T                                   [M, N] */
  SSA_EPILOGUE_RESIDUAL = 1, /* out = x W^T + residual                        [M, N] */
  SSA_EPILOGUE_SWIGLU = 2    /* out = silu(x Wg^T) * (x Wu^T)                 [M, N/2] */
};

/*
 * A linear layer on the matrix cores: out = x W^T with fp32 accumulation and
 * one bf16 rounding of the result (after the epilogue's fp32 arithmetic).
 *   x    [M, K] bf16, row-major;  W [N, K] bf16, row-major (torch Linear layout)
 *   out  [M, N] bf16 ([M, N/2] for SWIGLU); residual [M, N] bf16 (RESIDUAL only;
 *        it may be the same buffer as out)
 *   SWIGLU: W holds the gate and up projections interleaved in blocks of 16 rows
 *        (rows 32b .. 32b+15 = gate rows 16b .. 16b+15, rows 32b+16 .. 32b+31 =
 *        up rows 16b .. 16b+15); silu(z) = z / (1 + e^-z).
 *   workspace: ssa_linear_workspace_size bytes (0 when one pass over K fills the
 *        chip).  Its first words are split tickets: zero before the first call
 *        (a zeroed allocation), and zero again after every call.  Calls that
 *        share a workspace must be ordered on one stream.
 * Requires N % 128 == 0 and K % 64 == 0; M >= 0 (M == 0 does nothing); M K and N K
 * below 2^40 and (M / 32 + 1) (N / 128) at most 2^24.
 * Results do not depend on the launch order of workgroups: split partials are
 * added in split order.
 * Errors: SSA_ERR_ARG (sizes, epilogue), SSA_ERR_NULL, SSA_ERR_WORKSPACE,
 * SSA_ERR_HIP.
 */
int ssa_linear_workspace_size(int32_t m, int32_t n, int32_t k, size_t* ws_bytes);
int ssa_linear(int32_t m, int32_t n, int32_t k, int32_t epilogue, const uint16_t* x,
               const uint16_t* w, const uint16_t* residual, uint16_t* out, void* workspace,
               size_t ws_bytes, void* stream);

/*
 * RMSNorm of each row: out = x / sqrt(mean(x^2) + eps) * weight, in fp32, one
 * bf16 rounding.  x, out [M, N] bf16 (distinct buffers); weight [N] bf16.
 * Requires N % 8 == 0, N <= 8192, eps >= 0.
 * Errors: SSA_ERR_ARG, SSA_ERR_NULL, SSA_ERR_HIP.
 */
int ssa_rms_norm(int32_t m, int32_t n, const uint16_t* x, const uint16_t* weight, float eps,
                 uint16_t* out, void* stream);

/*
 * The weights of one Llama-style decoder layer (device pointers, bf16 unless
 * noted; the library keeps none of them).
 *   attn_norm, mlp_norm [hidden]          RMSNorm weights
 *   w_qkv     [(Hq + 2 Hkv) D, hidden]    query, key and value projections stacked
 *   w_o       [hidden, Hq D]              output projection
 *   w_gate_up [2 inter, hidden]           gate and up projections, interleaved in
 *                                         blocks of 16 rows (ssa_linear SWIGLU)
 *   w_down    [hidden, inter]             down projection
 *   cos_sin   [max_position, D] fp32      the rotary table of ssa_rope_append
 *   eps                                   the RMSNorm epsilon
 */
typedef struct ssa_layer_weights {
  const uint16_t* attn_norm;
  const uint16_t* w_qkv;
  const uint16_t* w_o;
  const uint16_t* mlp_norm;
  const uint16_t* w_gate_up;
  const uint16_t* w_down;
  const float* cos_sin;
  int32_t hidden, inter, max_position;
  float eps;
} ssa_layer_weights;

/*
 * Workspace bytes of ssa_layer_forward for this plan: the activations of the
 * plan's T tokens, the attention workspace of the plan, the linear layers'
 * split workspace.  The workspace must be zero before its first use (a zeroed
 * allocation); the counters in it are zero again after every call.
 */
int ssa_layer_workspace_size(const ssa_shape* shape, const void* plan_host,
                             const ssa_layer_weights* w, size_t* ws_bytes);

/*
 * One decoder layer over the T new tokens of a serving iteration (the batch
 * B = {(c_i, u_i)} of Sec. 3.2, Llama-3-8B's block, eight launches on `stream`):
 *   xn  = RMSNorm(x, attn_norm)
 *   qkv = xn w_qkv^T;  RoPE + kv_append (ssa_rope_append) -> q, the caches
 *   a   = ssa_mixed_attention(q, caches)
 *   h   = x + a w_o^T
 *   out = h + (silu(hn w_gate^T) * (hn w_up^T)) w_down^T,  hn = RMSNorm(h, mlp_norm)
 *   x, out [T, hidden] bf16, rows in plan order; out may be the same buffer as x.
 *   k_cache, v_cache, block_table: as ssa_kv_append (the new tokens' rotated
 *   keys and values are appended).
 * Requires hidden % 128 == 0, hidden <= 8192, inter % 64 == 0,
 * (Hq + 2 Hkv) D % 128 == 0.  Everything is validated before the first launch.
 * Errors: those of the steps (SSA_ERR_ARG for sizes and positions past the
 * rotary table), SSA_ERR_WORKSPACE, SSA_ERR_NULL, SSA_ERR_HIP.
 */
int ssa_layer_forward(const ssa_shape* shape, const void* plan_host, const void* plan_dev,
                      const ssa_layer_weights* w, const uint16_t* x, uint16_t* out,
                      uint16_t* k_cache, uint16_t* v_cache, const int32_t* block_table,
                      void* workspace, size_t ws_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SSA_LAYER_H */
