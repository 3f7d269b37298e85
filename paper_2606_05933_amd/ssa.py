"""Thin ctypes binding of ``libssa.so`` (declared in ``include/ssa.h``).

Argument marshalling only: every step of the attention path runs in the
library's host planner and HIP kernels.  The functions carry the C names.
Device arrays are torch tensors (``torch.bfloat16`` or 16-bit integer views for
bf16 data, ``torch.int32`` for the block table, ``torch.uint8`` for the plan
copy and the workspace); shapes are checked here against the layouts in
``ssa.h`` so that no launch can index outside a buffer it was given.

The library must be built (``paper_2606_05933_amd.build``); importing this
module without it raises - there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libssa.so")

SSA_OK = 0
SSA_ERR_NULL, SSA_ERR_WORKSPACE, SSA_ERR_HIP, SSA_ERR_ARG = -1, -8, -10, -13
SSA_ERR_PLAN_MISMATCH = -9
# the workspace's status word (ssa.h): byte offset and error bits
SSA_WS_STATUS_OFFSET = 8
SSA_STATUS_WAIT_TIMEOUT, SSA_STATUS_PLAN_MISMATCH = 1, 2
# workspace words ahead of the merge tickets (two counters, the status word, one spare)
WS_LAUNCH_WORDS = 4
SCENES = {0: "empty", 1: "pure decode", 2: "pure prefill", 3: "mixed"}


class SsaError(RuntimeError):
    def __init__(self, code: int, what: str):
        super().__init__(f"{what}: {ssa_status_string(code)} ({code})")
        self.code = code


class SsaShape(ctypes.Structure):
    _fields_ = [("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("page_size", ctypes.c_int32),
                ("num_pages", ctypes.c_int32), ("max_pages_per_req", ctypes.c_int32),
                ("softmax_scale", ctypes.c_float)]


class SsaTuning(ctypes.Structure):
    _fields_ = [("chunk_tile_cols", ctypes.c_int32), ("chunk_split_keys", ctypes.c_int32),
                ("decode_split_keys", ctypes.c_int32), ("num_cus", ctypes.c_int32),
                ("num_xcds", ctypes.c_int32), ("mix_order", ctypes.c_int32),
                ("append_wait_polls", ctypes.c_int32)]


PRED_FEATURES, PRED_MODELS, PRED_MOMENTS = 7, 4, 45


class SsaPredictor(ctypes.Structure):
    """ssa_predictor (include/ssa_predictor.h): caller-owned plain data."""
    _fields_ = [("samples", ctypes.c_int64 * PRED_MODELS),
                ("moments", (ctypes.c_double * PRED_MOMENTS) * PRED_MODELS),
                ("coef", (ctypes.c_double * (1 + PRED_FEATURES)) * PRED_MODELS),
                ("fitted", ctypes.c_int32 * PRED_MODELS),
                ("min_scene_samples", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class SsaPrefillRequest(ctypes.Structure):
    """ssa_prefill_request (include/ssa_chunker.h)."""
    _fields_ = [("cached", ctypes.c_int32), ("remaining", ctypes.c_int32)]


class SsaCandidate(ctypes.Structure):
    """ssa_candidate (include/ssa_constructor.h)."""
    _fields_ = [("cached", ctypes.c_int32), ("remaining", ctypes.c_int32),
                ("slack", ctypes.c_double), ("safeguard", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]


CONSTRUCT_NO_RISK, CONSTRUCT_NO_ANCHOR, CONSTRUCT_BATCH = 0, 1, 2


class SsaLayerWeights(ctypes.Structure):
    _fields_ = [("attn_norm", ctypes.c_void_p), ("w_qkv", ctypes.c_void_p),
                ("w_o", ctypes.c_void_p), ("mlp_norm", ctypes.c_void_p),
                ("w_gate_up", ctypes.c_void_p), ("w_down", ctypes.c_void_p),
                ("cos_sin", ctypes.c_void_p), ("hidden", ctypes.c_int32),
                ("inter", ctypes.c_int32), ("max_position", ctypes.c_int32),
                ("eps", ctypes.c_float)]


class SsaPlanInfo(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "num_reqs", "num_tokens", "num_decode_reqs", "num_chunk_reqs", "num_items",
        "num_chunk_items", "num_decode_items", "num_merge_groups", "num_append_segments",
        "scene")] + [(n, ctypes.c_double) for n in (
            "decode_bytes", "chunk_bytes", "chunk_flops", "decode_flops", "append_bytes")] + [
        ("x", ctypes.c_double * 7), ("ws_zero_bytes", ctypes.c_int64)]

    def as_dict(self):
        d = {n: getattr(self, n) for n, _ in self._fields_ if n != "x"}
        d["x"] = list(self.x)
        d["scene_name"] = SCENES.get(self.scene, "?")
        return d


def hip_runtimes_loaded() -> list[str]:
    """Distinct files of the HIP runtime (libamdhip64) mapped into this process."""
    paths = set()
    try:
        with open("/proc/self/maps") as f:
            for line in f:
                path = line.split()[-1] if line.strip() else ""
                if "libamdhip64" in os.path.basename(path):
                    paths.add(os.path.realpath(path))
    except OSError:
        pass
    return sorted(paths)


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run paper_2606_05933_amd.build.build() "
                          "(there is no non-HIP fallback)")
    # The library must share torch's HIP runtime: torch owns the device
    # memory and the streams it is called with.  torch loads its own copy of
    # libamdhip64 by file name; the library asks for the runtime by soname,
    # which resolves to torch's copy only if that is loaded first.  Loaded the
    # other way round, the process holds two runtimes, and a stream handle of
    # one is not valid in the other (every launch fails).
    import torch  # noqa: F401
    lib = ctypes.CDLL(LIB_PATH)
    runtimes = hip_runtimes_loaded()
    if len(runtimes) > 1:
        raise ImportError("more than one HIP runtime is loaded in this process: "
                          + ", ".join(runtimes)
                          + "; load libssa.so only after torch (import torch first)")
    vp, sz = ctypes.c_void_p, ctypes.c_size_t
    P = ctypes.POINTER
    lib.ssa_rope_table.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_double, vp]
    lib.ssa_rope_table.restype = ctypes.c_int
    lib.ssa_status_string.argtypes = [ctypes.c_int]
    lib.ssa_status_string.restype = ctypes.c_char_p
    lib.ssa_plan_size.argtypes = [P(SsaShape), vp, vp, ctypes.c_int32, P(SsaTuning), P(sz), P(sz)]
    lib.ssa_plan_size.restype = ctypes.c_int
    lib.ssa_plan.argtypes = [P(SsaShape), vp, vp, ctypes.c_int32, P(SsaTuning), vp, sz,
                             P(SsaPlanInfo)]
    lib.ssa_plan.restype = ctypes.c_int
    lib.ssa_kv_append.argtypes = [P(SsaShape), vp, vp, vp, vp, vp, vp, vp, vp]
    lib.ssa_kv_append.restype = ctypes.c_int
    lib.ssa_mixed_attention.argtypes = [P(SsaShape), vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.ssa_mixed_attention.restype = ctypes.c_int
    lib.ssa_kv_append_timed.argtypes = [P(SsaShape), vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    lib.ssa_kv_append_timed.restype = ctypes.c_int
    lib.ssa_mixed_attention_timed.argtypes = [P(SsaShape), vp, vp, vp, vp, vp, vp, vp, vp, sz, vp,
                                              vp, vp]
    lib.ssa_mixed_attention_timed.restype = ctypes.c_int
    lib.ssa_append_attention.argtypes = [P(SsaShape), vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz,
                                         vp, vp, vp]
    lib.ssa_append_attention.restype = ctypes.c_int
    lib.ssa_append_attention_static.argtypes = [P(SsaShape), vp, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                                vp, vp]
    lib.ssa_append_attention_static.restype = ctypes.c_int
    lib.ssa_append_attention_streams.argtypes = [P(SsaShape), vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                                 vp, sz, vp, vp, vp, vp]
    lib.ssa_append_attention_streams.restype = ctypes.c_int
    dp = P(ctypes.c_double)
    lib.ssa_predictor_init.argtypes = [P(SsaPredictor), ctypes.c_int32]
    lib.ssa_predictor_add.argtypes = [P(SsaPredictor), dp, ctypes.c_int32, ctypes.c_double]
    lib.ssa_predictor_fit.argtypes = [P(SsaPredictor)]
    lib.ssa_predictor_predict.argtypes = [P(SsaPredictor), dp, ctypes.c_int32, dp]
    ip, i32 = P(ctypes.c_int32), ctypes.c_int32
    lib.ssa_form_batch.argtypes = [ip, i32, P(SsaPrefillRequest), i32, i32, i32, ip, dp, ip]
    lib.ssa_time_to_budget.argtypes = [P(SsaPredictor), ip, i32, P(SsaPrefillRequest), i32, i32,
                                       ctypes.c_double, ip]
    lib.ssa_sliding_chunker.argtypes = [P(SsaPredictor), ip, i32, P(SsaPrefillRequest), i32, i32,
                                        ctypes.c_double, ctypes.c_double, ip, ip, dp]
    lib.ssa_rope_append.argtypes = [P(SsaShape), vp, vp, vp, vp, i32, vp, vp, vp, vp, vp]
    lib.ssa_rope_append.restype = ctypes.c_int
    lib.ssa_linear_workspace_size.argtypes = [i32, i32, i32, P(sz)]
    lib.ssa_linear.argtypes = [i32, i32, i32, i32, vp, vp, vp, vp, vp, sz, vp]
    lib.ssa_rms_norm.argtypes = [i32, i32, vp, vp, ctypes.c_float, vp, vp]
    lib.ssa_check_block_table.argtypes = [P(SsaShape), vp, vp]
    lib.ssa_v_pool_convert.argtypes = [P(SsaShape), vp, vp, i32, vp]
    lib.ssa_v_pool_convert.restype = ctypes.c_int
    lib.ssa_probe_hbm_read.argtypes = [vp, sz, vp, i32, vp]
    lib.ssa_probe_hbm_gather.argtypes = [vp, sz, vp, i32, i32, i32, vp, i32, vp]
    lib.ssa_probe_mfma_bf16.argtypes = [i32, i32, vp, vp]
    lib.ssa_layer_workspace_size.argtypes = [P(SsaShape), vp, P(SsaLayerWeights), P(sz)]
    lib.ssa_layer_forward.argtypes = [P(SsaShape), vp, vp, P(SsaLayerWeights), vp, vp, vp, vp, vp,
                                      vp, sz, vp]
    lib.ssa_priority_sort.argtypes = [P(SsaCandidate), i32, ctypes.c_double, ctypes.c_double,
                                      ctypes.c_double, ip]
    lib.ssa_batch_constructor.argtypes = [P(SsaPredictor), ip, i32, P(SsaCandidate), i32, i32,
                                          ctypes.c_double, ip, ip, ip, dp]
    for f in ("ssa_predictor_init", "ssa_predictor_add", "ssa_predictor_fit",
              "ssa_predictor_predict", "ssa_form_batch", "ssa_time_to_budget",
              "ssa_sliding_chunker", "ssa_priority_sort", "ssa_batch_constructor"):
        getattr(lib, f).restype = ctypes.c_int
    return lib


LIB = _load()

EXPORTED = ("ssa_status_string", "ssa_plan_size", "ssa_plan", "ssa_check_block_table",
            "ssa_v_pool_convert", "ssa_kv_append",
            "ssa_mixed_attention", "ssa_kv_append_timed", "ssa_mixed_attention_timed",
            "ssa_append_attention", "ssa_append_attention_static",
            "ssa_append_attention_streams", "ssa_predictor_init",
            "ssa_predictor_add",
            "ssa_predictor_fit", "ssa_predictor_predict", "ssa_form_batch", "ssa_time_to_budget",
            "ssa_sliding_chunker", "ssa_priority_sort", "ssa_batch_constructor",
            "ssa_rope_append", "ssa_rope_table", "ssa_linear_workspace_size", "ssa_linear", "ssa_rms_norm",
            "ssa_layer_workspace_size", "ssa_layer_forward", "ssa_probe_hbm_read",
            "ssa_probe_hbm_gather", "ssa_probe_mfma_bf16")

EPILOGUE_NONE, EPILOGUE_RESIDUAL, EPILOGUE_SWIGLU = 0, 1, 2


def _check(rc: int, what: str):
    if rc != 0:
        raise SsaError(rc, what)


class Predictor:
    """Batch latency predictor (Sec. 3.2, Eq. 5): argument marshalling around
    ssa_predictor_*; every step runs in the library."""

    def __init__(self, min_scene_samples: int = 16):
        self.p = SsaPredictor()
        _check(LIB.ssa_predictor_init(ctypes.byref(self.p), int(min_scene_samples)),
               "ssa_predictor_init")

    @staticmethod
    def _x(x):
        a = (ctypes.c_double * PRED_FEATURES)(*[float(v) for v in x])
        if len(x) != PRED_FEATURES:
            raise ValueError(f"{PRED_FEATURES} features expected")
        return a

    def add(self, x, scene: int, latency: float):
        _check(LIB.ssa_predictor_add(ctypes.byref(self.p), self._x(x), int(scene),
                                     float(latency)), "ssa_predictor_add")

    def fit(self):
        _check(LIB.ssa_predictor_fit(ctypes.byref(self.p)), "ssa_predictor_fit")
        return self

    def predict(self, x, scene: int) -> float:
        out = ctypes.c_double()
        _check(LIB.ssa_predictor_predict(ctypes.byref(self.p), self._x(x), int(scene),
                                         ctypes.byref(out)), "ssa_predictor_predict")
        return out.value

    def coefficients(self, model: int):
        """(b, w1..w7) of model 0 (global) or a scene, or None if not fitted."""
        if not self.p.fitted[model]:
            return None
        return np.array(list(self.p.coef[model]), dtype=np.float64)

    def copy(self) -> "Predictor":
        q = Predictor.__new__(Predictor)
        q.p = SsaPredictor()
        ctypes.memmove(ctypes.byref(q.p), ctypes.byref(self.p), ctypes.sizeof(SsaPredictor))
        return q


def _queue(decode_ctx, prefill):
    """(decode context lengths, [(cached, remaining), ...]) as C arrays."""
    dctx = (ctypes.c_int32 * max(1, len(decode_ctx)))(*[int(v) for v in decode_ctx])
    pf = (SsaPrefillRequest * max(1, len(prefill)))(
        *[SsaPrefillRequest(int(c), int(r)) for c, r in prefill])
    return dctx, len(decode_ctx), pf, len(prefill)


def form_batch(decode_ctx, prefill, budget: int, max_budget: int):
    """The batch a budget forms (Alg. 1's BatchForwarder): per-prefill chunks,
    Tab. 1 features, Eq. 3 scene."""
    dctx, nd, pf, npf = _queue(decode_ctx, prefill)
    chunk = (ctypes.c_int32 * max(1, npf))()
    x = (ctypes.c_double * PRED_FEATURES)()
    scene = ctypes.c_int32()
    _check(LIB.ssa_form_batch(dctx, nd, pf, npf, int(budget), int(max_budget), chunk, x,
                              ctypes.byref(scene)), "ssa_form_batch")
    return list(chunk)[:npf], list(x), scene.value


def time_to_budget(pred: Predictor, decode_ctx, prefill, max_budget: int, t_limit: float) -> int:
    dctx, nd, pf, npf = _queue(decode_ctx, prefill)
    out = ctypes.c_int32()
    _check(LIB.ssa_time_to_budget(ctypes.byref(pred.p), dctx, nd, pf, npf, int(max_budget),
                                  float(t_limit), ctypes.byref(out)), "ssa_time_to_budget")
    return out.value


def _candidates(cands):
    """[(cached, remaining, slack, safeguard), ...] as a C array."""
    return (SsaCandidate * max(1, len(cands)))(
        *[SsaCandidate(int(c), int(r), float(s), int(g), 0) for c, r, s, g in cands])


def priority_sort(cands, throughput: float, alpha: float, eps: float):
    """Eq. 12-13: candidate indices in priority order."""
    arr = _candidates(cands)
    order = (ctypes.c_int32 * max(1, len(cands)))()
    _check(LIB.ssa_priority_sort(arr, len(cands), float(throughput), float(alpha), float(eps),
                                 order), "ssa_priority_sort")
    return list(order)[:len(cands)]


def batch_constructor(pred: Predictor, decode_ctx, cands, max_budget: int, eps: float):
    """Alg. 2 on candidates in priority order: (outcome, budget, per-candidate
    tokens, predicted latency of the full batch); budget and tokens are None
    unless the outcome is CONSTRUCT_BATCH."""
    dctx = (ctypes.c_int32 * max(1, len(decode_ctx)))(*[int(v) for v in decode_ctx])
    arr = _candidates(cands)
    outcome, budget, tf = ctypes.c_int32(), ctypes.c_int32(-1), ctypes.c_double()
    take = (ctypes.c_int32 * max(1, len(cands)))()
    _check(LIB.ssa_batch_constructor(ctypes.byref(pred.p), dctx, len(decode_ctx), arr, len(cands),
                                     int(max_budget), float(eps), ctypes.byref(outcome),
                                     ctypes.byref(budget), take, ctypes.byref(tf)),
           "ssa_batch_constructor")
    if outcome.value != CONSTRUCT_BATCH:
        return outcome.value, None, None, tf.value
    return outcome.value, budget.value, list(take)[:len(cands)], tf.value


def sliding_chunker(pred: Predictor, decode_ctx, prefill, max_budget: int, t_cur: float,
                    t_next: float):
    """Alg. 1: (budget, per-prefill chunks, predicted latency of this iteration)."""
    dctx, nd, pf, npf = _queue(decode_ctx, prefill)
    budget = ctypes.c_int32()
    chunk = (ctypes.c_int32 * max(1, npf))()
    t = ctypes.c_double()
    _check(LIB.ssa_sliding_chunker(ctypes.byref(pred.p), dctx, nd, pf, npf, int(max_budget),
                                   float(t_cur), float(t_next), ctypes.byref(budget), chunk,
                                   ctypes.byref(t)), "ssa_sliding_chunker")
    return budget.value, list(chunk)[:npf], t.value


def ssa_status_string(code: int) -> str:
    return LIB.ssa_status_string(int(code)).decode()


def make_shape(hq, hkv, d, num_pages, max_pages_per_req, scale, page_size=16) -> SsaShape:
    return SsaShape(int(hq), int(hkv), int(d), int(page_size), int(num_pages),
                    int(max_pages_per_req), float(np.float32(scale)))


def make_tuning(chunk_tile_cols=0, chunk_split_keys=0, decode_split_keys=0, num_cus=0,
                num_xcds=0, mix_order=0, append_wait_polls=0):
    return SsaTuning(int(chunk_tile_cols), int(chunk_split_keys), int(decode_split_keys),
                     int(num_cus), int(num_xcds), int(mix_order), int(append_wait_polls))


def _lens(a):
    a = np.ascontiguousarray(np.asarray(a, dtype=np.int32).reshape(-1))
    return a, (a.ctypes.data if a.size else None)


def ssa_plan_size(shape: SsaShape, q_len, ctx_len, tuning: SsaTuning | None = None):
    ql, pq = _lens(q_len)
    cl, pc = _lens(ctx_len)
    if ql.shape != cl.shape:
        raise ValueError("q_len and ctx_len differ in length")
    pb, wb = ctypes.c_size_t(), ctypes.c_size_t()
    rc = LIB.ssa_plan_size(ctypes.byref(shape), pq, pc, ql.shape[0],
                           ctypes.byref(tuning) if tuning is not None else None,
                           ctypes.byref(pb), ctypes.byref(wb))
    if rc != SSA_OK:
        raise SsaError(rc, "ssa_plan_size")
    return pb.value, wb.value


def ssa_plan(shape: SsaShape, q_len, ctx_len, tuning: SsaTuning | None = None, out=None):
    """Plan blob (numpy uint8, or written into ``out``: a host buffer exposing
    ``data_ptr()``/``numel()`` or a numpy array) and the plan info."""
    ql, pq = _lens(q_len)
    cl, pc = _lens(ctx_len)
    nbytes, _ = ssa_plan_size(shape, ql, cl, tuning)
    if out is None:
        out = np.zeros(nbytes, dtype=np.uint8)
    if isinstance(out, np.ndarray):
        ptr, cap = out.ctypes.data, out.nbytes
    else:
        ptr, cap = out.data_ptr(), out.numel() * out.element_size()
    info = SsaPlanInfo()
    rc = LIB.ssa_plan(ctypes.byref(shape), pq, pc, ql.shape[0],
                      ctypes.byref(tuning) if tuning is not None else None, ptr, cap,
                      ctypes.byref(info))
    if rc != SSA_OK:
        raise SsaError(rc, "ssa_plan")
    return out, info


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, np.ndarray):
        return x.ctypes.data
    return x.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return getattr(stream, "cuda_stream", stream)


def _check_dev(name, t, numel, itemsize):
    if t is None:
        return
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.element_size() != itemsize:
        raise ValueError(f"{name} must have {itemsize}-byte elements")
    if t.numel() < numel:
        raise ValueError(f"{name} holds {t.numel()} elements, the layout needs {numel}")


def _plan_header(plan_host):
    h = np.frombuffer(bytes(np.asarray(_as_np(plan_host))[:128]), dtype=np.int32)
    return {"num_reqs": int(h[4]), "num_tokens": int(h[5]), "num_items": int(h[6]),
            "num_segments": int(h[10])}


def _as_np(plan_host):
    if isinstance(plan_host, np.ndarray):
        return plan_host
    return plan_host.numpy()


def ssa_kv_append(shape: SsaShape, plan_host, plan_dev, k_new, v_new, k_cache, v_cache,
                  block_table, stream=None):
    h = _plan_header(plan_host)
    T, n = h["num_tokens"], h["num_reqs"]
    row = shape.num_kv_heads * shape.head_dim
    pool = shape.num_pages * shape.num_kv_heads * shape.page_size * shape.head_dim
    _check_dev("k_new", k_new, T * row, 2)
    _check_dev("v_new", v_new, T * row, 2)
    _check_dev("k_cache", k_cache, pool, 2)
    _check_dev("v_cache", v_cache, pool, 2)
    _check_dev("block_table", block_table, n * shape.max_pages_per_req, 4)
    rc = LIB.ssa_kv_append(ctypes.byref(shape), _ptr(plan_host), _ptr(plan_dev), _ptr(k_new),
                           _ptr(v_new), _ptr(k_cache), _ptr(v_cache), _ptr(block_table),
                           _stream(stream))
    if rc != SSA_OK:
        raise SsaError(rc, "ssa_kv_append")


def ssa_mixed_attention(shape: SsaShape, plan_host, plan_dev, q, k_cache, v_cache, block_table,
                        out, workspace, stream=None):
    h = _plan_header(plan_host)
    T, n = h["num_tokens"], h["num_reqs"]
    qrow = shape.num_q_heads * shape.head_dim
    pool = shape.num_pages * shape.num_kv_heads * shape.page_size * shape.head_dim
    _check_dev("q", q, T * qrow, 2)
    _check_dev("out", out, T * qrow, 2)
    _check_dev("k_cache", k_cache, pool, 2)
    _check_dev("v_cache", v_cache, pool, 2)
    _check_dev("block_table", block_table, n * shape.max_pages_per_req, 4)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    rc = LIB.ssa_mixed_attention(ctypes.byref(shape), _ptr(plan_host), _ptr(plan_dev), _ptr(q),
                                 _ptr(k_cache), _ptr(v_cache), _ptr(block_table), _ptr(out),
                                 _ptr(workspace), ws_bytes, _stream(stream))
    if rc != SSA_OK:
        raise SsaError(rc, "ssa_mixed_attention")


class BoundCall:
    """A C entry point with its arguments checked and marshalled once, for a
    serving loop that repeats the same call (same buffers, same plan buffer)
    every iteration.  Calling it only crosses into the library."""

    def __init__(self, fn, name, args, timed=False):
        self._fn, self._name, self._args = fn, name, args
        self._untimed = args + (None, None) if timed else args

    def __call__(self, start_event=None, stop_event=None):
        """start_event / stop_event (timed entry points only): torch.cuda.Event
        objects (timing enabled, recorded at least once so that the HIP event
        exists) that receive the kernel's own start and end times."""
        if start_event is None and stop_event is None:
            rc = self._fn(*self._untimed)
        else:
            rc = self._fn(*self._args, _event(start_event), _event(stop_event))
        if rc != SSA_OK:
            raise SsaError(rc, self._name)


def _event(ev):
    if ev is None:
        return None
    handle = ev.cuda_event
    if not handle:
        raise ValueError("the event has no HIP event yet: record it once before timing")
    return ctypes.c_void_p(handle)


def bind_kv_append(shape: SsaShape, plan_host, plan_dev, k_new, v_new, k_cache, v_cache,
                   block_table, stream=None) -> BoundCall:
    h = _plan_header(plan_host)
    T, n = h["num_tokens"], h["num_reqs"]
    row = shape.num_kv_heads * shape.head_dim
    pool = shape.num_pages * shape.num_kv_heads * shape.page_size * shape.head_dim
    _check_dev("k_new", k_new, T * row, 2)
    _check_dev("v_new", v_new, T * row, 2)
    _check_dev("k_cache", k_cache, pool, 2)
    _check_dev("v_cache", v_cache, pool, 2)
    _check_dev("block_table", block_table, n * shape.max_pages_per_req, 4)
    vp = ctypes.c_void_p
    args = (ctypes.byref(shape), vp(_ptr(plan_host)), vp(_ptr(plan_dev)), vp(_ptr(k_new)),
            vp(_ptr(v_new)), vp(_ptr(k_cache)), vp(_ptr(v_cache)), vp(_ptr(block_table)),
            vp(_stream(stream)))
    return BoundCall(LIB.ssa_kv_append_timed, "ssa_kv_append", args, timed=True)


def bind_mixed_attention(shape: SsaShape, plan_host, plan_dev, q, k_cache, v_cache, block_table,
                         out, workspace, stream=None) -> BoundCall:
    h = _plan_header(plan_host)
    T, n = h["num_tokens"], h["num_reqs"]
    qrow = shape.num_q_heads * shape.head_dim
    pool = shape.num_pages * shape.num_kv_heads * shape.page_size * shape.head_dim
    _check_dev("q", q, T * qrow, 2)
    _check_dev("out", out, T * qrow, 2)
    _check_dev("k_cache", k_cache, pool, 2)
    _check_dev("v_cache", v_cache, pool, 2)
    _check_dev("block_table", block_table, n * shape.max_pages_per_req, 4)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    vp = ctypes.c_void_p
    args = (ctypes.byref(shape), vp(_ptr(plan_host)), vp(_ptr(plan_dev)), vp(_ptr(q)),
            vp(_ptr(k_cache)), vp(_ptr(v_cache)), vp(_ptr(block_table)), vp(_ptr(out)),
            vp(_ptr(workspace)), ctypes.c_size_t(ws_bytes), vp(_stream(stream)))
    return BoundCall(LIB.ssa_mixed_attention_timed, "ssa_mixed_attention", args, timed=True)


def rope_cos_sin(max_position: int, d: int, base: float = 500000.0) -> np.ndarray:
    """[max_position, d] fp32 table of ssa_rope_append (ssa_rope_table): cos(p t_i)
    in columns i < d/2, sin(p t_i) in columns d/2 + i, t_i = base^(-2i/d)."""
    out = np.empty((max_position, d), dtype=np.float32)
    rc = LIB.ssa_rope_table(int(max_position), int(d), float(base), out.ctypes.data)
    if rc != SSA_OK:
        raise SsaError(rc, "ssa_rope_table")
    return out


def rope_append(shape: SsaShape, plan_host, plan_dev, qkv, cos_sin, q_out, k_cache, v_cache,
                block_table, stream=None):
    """ssa_rope_append: RoPE of the new queries and keys, and kv_append of the
    rotated keys and the values, in one launch."""
    h = _plan_header(plan_host)
    T, n = h["num_tokens"], h["num_reqs"]
    d, hq, hkv = shape.head_dim, shape.num_q_heads, shape.num_kv_heads
    pool = shape.num_pages * hkv * shape.page_size * d
    _check_dev("qkv", qkv, T * (hq + 2 * hkv) * d, 2)
    _check_dev("q_out", q_out, T * hq * d, 2)
    _check_dev("cos_sin", cos_sin, d, 4)
    _check_dev("k_cache", k_cache, pool, 2)
    _check_dev("v_cache", v_cache, pool, 2)
    _check_dev("block_table", block_table, n * shape.max_pages_per_req, 4)
    max_pos = cos_sin.numel() // d
    vp = ctypes.c_void_p
    rc = LIB.ssa_rope_append(ctypes.byref(shape), vp(_ptr(plan_host)), vp(_ptr(plan_dev)),
                             vp(_ptr(qkv)), vp(_ptr(cos_sin)), int(max_pos), vp(_ptr(q_out)),
                             vp(_ptr(k_cache)), vp(_ptr(v_cache)), vp(_ptr(block_table)),
                             vp(_stream(stream)))
    if rc != SSA_OK:
        raise SsaError(rc, "ssa_rope_append")


def linear_workspace_size(m: int, n: int, k: int) -> int:
    """Bytes of the workspace ssa_linear needs for an [m, k] x [n, k]^T product."""
    ws = ctypes.c_size_t(0)
    _check(LIB.ssa_linear_workspace_size(int(m), int(n), int(k), ctypes.byref(ws)),
           "ssa_linear_workspace_size")
    return int(ws.value)


def linear(x, w, out, epilogue: int = EPILOGUE_NONE, residual=None, workspace=None, stream=None):
    """ssa_linear: out = x w^T (+ residual, or the SwiGLU of interleaved gate/up
    rows), x [m, k], w [n, k], bf16 device tensors."""
    m, k = x.shape[0], x.shape[-1]
    n = w.shape[0]
    _check_dev("x", x, m * k, 2)
    _check_dev("w", w, n * k, 2)
    _check_dev("out", out, m * (n // 2 if epilogue == EPILOGUE_SWIGLU else n), 2)
    if epilogue == EPILOGUE_RESIDUAL:
        _check_dev("residual", residual, m * n, 2)
    if w.numel() != n * k or x.numel() != m * k:
        raise ValueError("x and w must be [m, k] and [n, k]")
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    vp = ctypes.c_void_p
    rc = LIB.ssa_linear(int(m), int(n), int(k), int(epilogue), vp(_ptr(x)), vp(_ptr(w)),
                        vp(_ptr(residual)), vp(_ptr(out)), vp(_ptr(workspace)),
                        ctypes.c_size_t(ws_bytes), vp(_stream(stream)))
    if rc != SSA_OK:
        raise SsaError(rc, "ssa_linear")


def v_pool_convert(shape: SsaShape, src, dst, to_dim_major: bool = True, stream=None):
    """ssa_v_pool_convert: a value pool [num_pages, Hkv, 16, D] -> [num_pages, Hkv, D, 16]
    (to_dim_major) or back, device tensors of 2-byte elements."""
    numel = shape.num_pages * shape.num_kv_heads * shape.page_size * shape.head_dim
    _check_dev("src", src, numel, 2)
    _check_dev("dst", dst, numel, 2)
    vp = ctypes.c_void_p
    rc = LIB.ssa_v_pool_convert(ctypes.byref(shape), vp(_ptr(src)), vp(_ptr(dst)),
                                int(bool(to_dim_major)), vp(_stream(stream)))
    if rc != SSA_OK:
        raise SsaError(rc, "ssa_v_pool_convert")


def rms_norm(x, weight, out, eps: float = 1e-5, stream=None):
    """ssa_rms_norm of each row of x [m, n] (bf16 device tensors)."""
    m, n = x.shape[0], x.shape[-1]
    _check_dev("x", x, m * n, 2)
    _check_dev("weight", weight, n, 2)
    _check_dev("out", out, m * n, 2)
    vp = ctypes.c_void_p
    rc = LIB.ssa_rms_norm(int(m), int(n), vp(_ptr(x)), vp(_ptr(weight)), ctypes.c_float(eps),
                          vp(_ptr(out)), vp(_stream(stream)))
    if rc != SSA_OK:
        raise SsaError(rc, "ssa_rms_norm")


def interleave_gate_up(w_gate, w_up):
    """The [2I, K] weight of ssa_linear's SwiGLU epilogue from the gate and up
    weights [I, K] (I % 64 == 0): blocks of 16 gate rows and 16 up rows
    alternate.  A one-time layout change of the weights (numpy or torch)."""
    i, k = w_gate.shape
    if w_up.shape != (i, k) or i % 16:
        raise ValueError("gate and up weights must both be [I, K] with I % 16 == 0")
    if isinstance(w_gate, np.ndarray):
        return np.stack([w_gate.reshape(i // 16, 16, k), w_up.reshape(i // 16, 16, k)],
                        axis=1).reshape(2 * i, k)
    import torch
    return torch.stack([w_gate.reshape(i // 16, 16, k), w_up.reshape(i // 16, 16, k)],
                       dim=1).reshape(2 * i, k).contiguous()


class LayerWeights:
    """Device copies of one decoder layer's weights in the layout of
    ssa_layer_forward (q/k/v rows stacked, gate/up rows interleaved), and the
    rotary table.  `host` holds bf16 bit arrays [out, in] (numpy uint16)."""

    def __init__(self, host: dict, hq: int, hkv: int, d: int, max_position: int,
                 eps: float = 1e-5, base: float = 500000.0):
        import torch

        def dev(bits):
            return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(
                torch.bfloat16)

        self.hidden = int(host["w_q"].shape[1])
        self.inter = int(host["w_gate"].shape[0])
        self.hq, self.hkv, self.d = hq, hkv, d
        self.attn_norm = dev(host["attn_norm"])
        self.mlp_norm = dev(host["mlp_norm"])
        self.w_qkv = dev(np.concatenate([host["w_q"], host["w_k"], host["w_v"]], axis=0))
        self.w_o = dev(host["w_o"])
        self.w_gate_up = dev(interleave_gate_up(host["w_gate"], host["w_up"]))
        self.w_down = dev(host["w_down"])
        self.cos_sin = torch.from_numpy(rope_cos_sin(max_position, d, base)).cuda()
        self.c = SsaLayerWeights(self.attn_norm.data_ptr(), self.w_qkv.data_ptr(),
                                 self.w_o.data_ptr(), self.mlp_norm.data_ptr(),
                                 self.w_gate_up.data_ptr(), self.w_down.data_ptr(),
                                 self.cos_sin.data_ptr(), self.hidden, self.inter,
                                 int(max_position), float(eps))


def check_block_table(shape: SsaShape, plan_host, block_table_host) -> None:
    """ssa_check_block_table on a host copy of the block table (int32 numpy
    array [num_reqs, max_pages_per_req]); raises SsaError on a bad entry and
    ValueError when the array does not have that shape (the library reads
    num_reqs rows of max_pages_per_req entries)."""
    bt = np.ascontiguousarray(block_table_host, dtype=np.int32)
    h = _plan_header(plan_host)
    if bt.ndim != 2 or bt.shape != (h["num_reqs"], shape.max_pages_per_req):
        raise ValueError(f"block table of shape {bt.shape}, the plan needs "
                         f"({h['num_reqs']}, {shape.max_pages_per_req})")
    _check(LIB.ssa_check_block_table(ctypes.byref(shape), ctypes.c_void_p(_ptr(plan_host)),
                                     ctypes.c_void_p(bt.ctypes.data)), "ssa_check_block_table")


def probe_hbm_read(src, out, workgroups: int, stream=None):
    """ssa_probe_hbm_read over the whole of the device tensor src."""
    nbytes = src.numel() * src.element_size()
    _check(LIB.ssa_probe_hbm_read(ctypes.c_void_p(_ptr(src)), ctypes.c_size_t(nbytes),
                                  ctypes.c_void_p(_ptr(out)), int(workgroups),
                                  ctypes.c_void_p(_stream(stream))), "ssa_probe_hbm_read")
    return nbytes


def probe_hbm_gather(src, chunk_index, chunk_bytes: int, out, workgroups: int, stream=None,
                     pattern: int = 0):
    """ssa_probe_hbm_gather of the chunks chunk_index (int32 device tensor) names
    in the device tensor src (pattern 1: the key rows' load pattern, 4 KB
    chunks); returns the bytes of the named chunks."""
    nbytes = src.numel() * src.element_size()
    _check_dev("chunk_index", chunk_index, chunk_index.numel(), 4)
    _check_dev("out", out, workgroups, 4)
    _check(LIB.ssa_probe_hbm_gather(ctypes.c_void_p(_ptr(src)), ctypes.c_size_t(nbytes),
                                    ctypes.c_void_p(_ptr(chunk_index)), int(chunk_index.numel()),
                                    int(chunk_bytes), int(pattern), ctypes.c_void_p(_ptr(out)),
                                    int(workgroups),
                                    ctypes.c_void_p(_stream(stream))), "ssa_probe_hbm_gather")
    return chunk_index.numel() * chunk_bytes


def probe_mfma_bf16(iters: int, workgroups: int, out, stream=None):
    """ssa_probe_mfma_bf16; returns the flops of the launch."""
    _check(LIB.ssa_probe_mfma_bf16(int(iters), int(workgroups), ctypes.c_void_p(_ptr(out)),
                                   ctypes.c_void_p(_stream(stream))), "ssa_probe_mfma_bf16")
    return workgroups * 4 * iters * 16 * 16384


def layer_workspace_size(shape: SsaShape, plan_host, weights: LayerWeights) -> int:
    ws = ctypes.c_size_t(0)
    _check(LIB.ssa_layer_workspace_size(ctypes.byref(shape), ctypes.c_void_p(_ptr(plan_host)),
                                        ctypes.byref(weights.c), ctypes.byref(ws)),
           "ssa_layer_workspace_size")
    return int(ws.value)


def layer_forward(shape: SsaShape, plan_host, plan_dev, weights: LayerWeights, x, out, k_cache,
                  v_cache, block_table, workspace, stream=None):
    """ssa_layer_forward: one decoder layer over the plan's new tokens (x, out
    [T, hidden] bf16; out may be x)."""
    h = _plan_header(plan_host)
    T, n = h["num_tokens"], h["num_reqs"]
    pool = shape.num_pages * shape.num_kv_heads * shape.page_size * shape.head_dim
    _check_dev("x", x, T * weights.hidden, 2)
    _check_dev("out", out, T * weights.hidden, 2)
    _check_dev("k_cache", k_cache, pool, 2)
    _check_dev("v_cache", v_cache, pool, 2)
    _check_dev("block_table", block_table, n * shape.max_pages_per_req, 4)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    vp = ctypes.c_void_p
    rc = LIB.ssa_layer_forward(ctypes.byref(shape), vp(_ptr(plan_host)), vp(_ptr(plan_dev)),
                               ctypes.byref(weights.c), vp(_ptr(x)), vp(_ptr(out)),
                               vp(_ptr(k_cache)), vp(_ptr(v_cache)), vp(_ptr(block_table)),
                               vp(_ptr(workspace)), ctypes.c_size_t(ws_bytes), vp(_stream(stream)))
    if rc != SSA_OK:
        raise SsaError(rc, "ssa_layer_forward")


def _check_fused_buffers(shape: SsaShape, plan_host, q, k_new, v_new, k_cache, v_cache,
                         block_table, out):
    h = _plan_header(plan_host)
    T, n = h["num_tokens"], h["num_reqs"]
    qrow = shape.num_q_heads * shape.head_dim
    row = shape.num_kv_heads * shape.head_dim
    pool = shape.num_pages * shape.num_kv_heads * shape.page_size * shape.head_dim
    _check_dev("q", q, T * qrow, 2)
    _check_dev("out", out, T * qrow, 2)
    _check_dev("k_new", k_new, T * row, 2)
    _check_dev("v_new", v_new, T * row, 2)
    _check_dev("k_cache", k_cache, pool, 2)
    _check_dev("v_cache", v_cache, pool, 2)
    _check_dev("block_table", block_table, n * shape.max_pages_per_req, 4)


def _fused_args(shape: SsaShape, plan_host, plan_dev, q, k_new, v_new, k_cache, v_cache,
                block_table, out, workspace):
    _check_fused_buffers(shape, plan_host, q, k_new, v_new, k_cache, v_cache, block_table, out)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    vp = ctypes.c_void_p
    return (ctypes.byref(shape), vp(_ptr(plan_host)), vp(_ptr(plan_dev)), vp(_ptr(q)),
            vp(_ptr(k_new)), vp(_ptr(v_new)), vp(_ptr(k_cache)), vp(_ptr(v_cache)),
            vp(_ptr(block_table)), vp(_ptr(out)), vp(_ptr(workspace)), ctypes.c_size_t(ws_bytes))


def bind_append_attention(shape: SsaShape, plan_host, plan_dev, q, k_new, v_new, k_cache, v_cache,
                          block_table, out, workspace, stream=None) -> BoundCall:
    """ssa_append_attention (kv_append and mixed attention in one launch);
    calling the result takes optional (start, stop) events."""
    args = _fused_args(shape, plan_host, plan_dev, q, k_new, v_new, k_cache, v_cache,
                       block_table, out, workspace)
    return BoundCall(LIB.ssa_append_attention, "ssa_append_attention",
                     args + (ctypes.c_void_p(_stream(stream)),), timed=True)


def bind_append_attention_streams(shape: SsaShape, plan_host, plan_dev, q, k_new, v_new, k_cache,
                                  v_cache, block_table, out, workspace, stream=None,
                                  decode_stream=None) -> BoundCall:
    """ssa_append_attention_streams (the chunk rows on `stream`, the decode rows
    beside them on `decode_stream`); the plan must list chunk items first
    (tuning mix_order = 1).  Calling the result takes optional (start, stop)
    events, recorded on `stream` around both launches."""
    args = _fused_args(shape, plan_host, plan_dev, q, k_new, v_new, k_cache, v_cache,
                       block_table, out, workspace)
    vp = ctypes.c_void_p
    return BoundCall(LIB.ssa_append_attention_streams, "ssa_append_attention_streams",
                     args + (vp(_stream(stream)), vp(_stream(decode_stream))), timed=True)


def append_attention_static(shape: SsaShape, plan_host, plan_dev, q, k_new, v_new, k_cache,
                            v_cache, block_table, out, stream=None, events=(None, None)):
    """ssa_append_attention_static: the fused launch with the library's own
    per-GPU scratch in place of a workspace (nothing is allocated)."""
    _check_fused_buffers(shape, plan_host, q, k_new, v_new, k_cache, v_cache, block_table, out)
    vp = ctypes.c_void_p
    start, stop = events
    _check(LIB.ssa_append_attention_static(
        ctypes.byref(shape), vp(_ptr(plan_host)), vp(_ptr(plan_dev)), vp(_ptr(q)),
        vp(_ptr(k_new)), vp(_ptr(v_new)), vp(_ptr(k_cache)), vp(_ptr(v_cache)),
        vp(_ptr(block_table)), vp(_ptr(out)), vp(_stream(stream)),
        vp(None if start is None else start.cuda_event),
        vp(None if stop is None else stop.cuda_event)), "ssa_append_attention_static")


def bind_plan(shape: SsaShape, q_len, ctx_len, tuning, out, info: SsaPlanInfo) -> BoundCall:
    """ssa_plan into a fixed host buffer (numpy array or pinned tensor)."""
    ql, pq = _lens(q_len)
    cl, pc = _lens(ctx_len)
    if isinstance(out, np.ndarray):
        ptr, cap = out.ctypes.data, out.nbytes
    else:
        ptr, cap = out.data_ptr(), out.numel() * out.element_size()
    vp = ctypes.c_void_p
    args = (ctypes.byref(shape), vp(pq), vp(pc), ctypes.c_int32(ql.shape[0]),
            ctypes.byref(tuning) if tuning is not None else None, vp(ptr), ctypes.c_size_t(cap),
            ctypes.byref(info))
    call = BoundCall(LIB.ssa_plan, "ssa_plan", args)
    call._keep = (ql, cl)  # the length arrays must outlive the call
    return call
