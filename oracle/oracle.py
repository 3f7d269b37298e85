"""Python front of the CPU oracle (``ssa_oracle.c``).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, the smoke check and the
benchmark's CPU-baseline leg, never by the library.  It takes plain numpy arrays
(bf16 as uint16 bit patterns) and imports nothing from the library package.

What is computed, and the layouts, are described at the top of ``ssa_oracle.c``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ssa_oracle.c")
_LIB = os.path.join(_HERE, "libssa_oracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (plain -O2, OpenMP, no fast-math)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
                               "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def bind(path: str):
    """Load an oracle shared object (the tests also load deliberately broken
    copies of it to show that the pins catch planted mistakes)."""
    lib = ctypes.CDLL(path)
    i32, f32, vp, i64 = ctypes.c_int, ctypes.c_float, ctypes.c_void_p, ctypes.c_int64
    lib.oracle_kv_append.argtypes = [i32, i32, i32, i32, vp, vp, vp, i32, vp, vp, vp, vp]
    lib.oracle_kv_append.restype = None
    lib.oracle_attention.argtypes = [i32, i32, i32, i32, f32, i32, vp, vp, vp, i32,
                                     vp, vp, vp, vp, i32]
    lib.oracle_attention.restype = ctypes.c_int
    lib.oracle_attention_rows.argtypes = [i32, i32, i32, i32, f32, i32, vp, vp, vp, i32,
                                          vp, vp, vp, vp, vp, i64, vp, i32]
    lib.oracle_attention_rows.restype = ctypes.c_int
    return lib


def _load(lib=None):
    global _lib
    if lib is not None:
        return lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        _lib = bind(_LIB)
    return _lib


def _c(a, dtype):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a, a.ctypes.data


def kv_append(hkv, d, page, q_len, ctx_len, block_table, k_new, v_new, k_cache, v_cache,
              lib=None):
    """Return copies of the pools after the append of this iteration's K/V rows."""
    lib = _load(lib)
    ql, pql = _c(q_len, np.int32)
    cl, pcl = _c(ctx_len, np.int32)
    bt, pbt = _c(block_table, np.int32)
    kn, pkn = _c(k_new, np.uint16)
    vn, pvn = _c(v_new, np.uint16)
    kc = np.array(k_cache, dtype=np.uint16, copy=True, order="C")
    vc = np.array(v_cache, dtype=np.uint16, copy=True, order="C")
    lib.oracle_kv_append(hkv, d, page, ql.shape[0], pql, pcl, pbt, bt.shape[1], pkn, pvn,
                         kc.ctypes.data, vc.ctypes.data)
    return kc, vc


def kv_append_inplace(hkv, d, page, q_len, ctx_len, block_table, k_new, v_new, k_cache,
                      v_cache, lib=None):
    """The same append, written into the given C-contiguous uint16 pools."""
    lib = _load(lib)
    for a in (k_cache, v_cache):
        if a.dtype != np.uint16 or not a.flags.c_contiguous:
            raise ValueError("pools must be C-contiguous uint16 arrays")
    ql, pql = _c(q_len, np.int32)
    cl, pcl = _c(ctx_len, np.int32)
    bt, pbt = _c(block_table, np.int32)
    kn, pkn = _c(k_new, np.uint16)
    vn, pvn = _c(v_new, np.uint16)
    lib.oracle_kv_append(hkv, d, page, ql.shape[0], pql, pcl, pbt, bt.shape[1], pkn, pvn,
                         k_cache.ctypes.data, v_cache.ctypes.data)


def attention(hq, hkv, d, page, scale, q_len, ctx_len, block_table, q, k_cache, v_cache,
              threads: int = 0, lib=None):
    """fp64 output [T, Hq, D] and the number of threads used."""
    lib = _load(lib)
    ql, pql = _c(q_len, np.int32)
    cl, pcl = _c(ctx_len, np.int32)
    bt, pbt = _c(block_table, np.int32)
    qq, pq = _c(q, np.uint16)
    kc, pk = _c(k_cache, np.uint16)
    vc, pv = _c(v_cache, np.uint16)
    T = int(ql.sum())
    out = np.zeros((T, hq, d), dtype=np.float64)
    used = lib.oracle_attention(hq, hkv, d, page, float(np.float32(scale)), ql.shape[0], pql,
                                pcl, pbt, bt.shape[1], pq, pk, pv, out.ctypes.data, int(threads))
    return out, used


def attention_rows(hq, hkv, d, page, scale, q_len, ctx_len, block_table, q, k_cache, v_cache,
                   rows, heads, threads: int = 0, lib=None):
    """fp64 outputs [n, D] at the selected (token row, q head) pairs."""
    lib = _load(lib)
    ql, pql = _c(q_len, np.int32)
    cl, pcl = _c(ctx_len, np.int32)
    bt, pbt = _c(block_table, np.int32)
    qq, pq = _c(q, np.uint16)
    kc, pk = _c(k_cache, np.uint16)
    vc, pv = _c(v_cache, np.uint16)
    r, pr = _c(rows, np.int64)
    h, ph = _c(heads, np.int32)
    out = np.zeros((r.shape[0], d), dtype=np.float64)
    used = lib.oracle_attention_rows(hq, hkv, d, page, float(np.float32(scale)), ql.shape[0],
                                     pql, pcl, pbt, bt.shape[1], pq, pk, pv, pr, ph, r.shape[0],
                                     out.ctypes.data, int(threads))
    return out, used


def batch_kv_append(b, lib=None):
    """kv_append for a batch object with the generator's field names."""
    s = b.shape
    return kv_append(s.hkv, s.d, s.page, b.q_len, b.ctx_len, b.block_table, b.k_new, b.v_new,
                     b.k_cache, b.v_cache, lib=lib)


def batch_attention(b, k_cache=None, v_cache=None, threads: int = 0, lib=None):
    """Oracle output of a batch whose pools already hold the appended rows
    (pass them in), or, by default, after appending them here."""
    if k_cache is None:
        k_cache, v_cache = batch_kv_append(b, lib=lib)
    s = b.shape
    return attention(s.hq, s.hkv, s.d, s.page, s.softmax_scale, b.q_len, b.ctx_len,
                     b.block_table, b.q, k_cache, v_cache, threads, lib=lib)
