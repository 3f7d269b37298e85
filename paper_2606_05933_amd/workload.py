"""Seeded synthetic batches for mixed chunked-prefill + decode paged attention.

This module only draws inputs.  It holds none of the attention arithmetic and is
the one piece of code that both the HIP path (through its tests, ``bench.py``
and ``smoke()``) and the CPU oracle consume.

A batch is the paper's iteration descriptor B = {(c_i, u_i)} (Sec. 3.2): for each
request, ``q_len[i]`` = c_i new tokens computed this iteration and
``ctx_len[i]`` = u_i tokens already in the KV cache.  Requests with c_i <= 1 are
the decode set D and the others the prefill set P (Sec. 3.2, Eq. 2); the
generator does not route, it only draws lengths and values.

Data layout (the boundary's contract, see ``include/ssa.h``):

* ``q``      bf16 ``[T, Hq, D]``, rows grouped by request in request order;
* ``k_new``  bf16 ``[T, Hkv, D]`` and ``v_new`` bf16 ``[T, Hkv, D]``;
* ``k_cache`` bf16 ``[num_pages, Hkv, P, D]``  (slot-major K page);
* ``v_cache`` bf16 ``[num_pages, Hkv, D, P]``  (dim-major V page);
* ``block_table`` int32 ``[num_reqs, max_pages_per_req]``, -1 past a request's
  last page.

bf16 values travel as ``uint16`` bit patterns (numpy has no bf16).  Every value
is an fp32 standard normal rounded to bf16 with round-to-nearest-even.  Pages
come from a seeded permutation of a pool that holds ``spare_pages`` more pages
than the batch needs.  Every pool slot that does not hold a cached token of some
request (slots at positions >= u_i, spare pages) is filled with a bf16 quiet NaN
when ``poison`` is set, so that a kernel that reads a key it must not see, or
multiplies a masked weight by such a slot, shows up as NaN.
"""
from __future__ import annotations

import concurrent.futures
import dataclasses
import hashlib
import math
import os

import numpy as np

PAGE_SIZE = 16
BF16_NAN = np.uint16(0x7FC0)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (round to nearest, ties to even); returns uint16 bits.

    Inputs here are finite normals, so the NaN/overflow corner of the rounding
    add never arises.
    """
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    b = u >> np.uint32(16)
    b &= np.uint32(1)
    b += np.uint32(0x7FFF)
    b += u
    b >>= np.uint32(16)
    return b.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


@dataclasses.dataclass(frozen=True)
class Shape:
    hq: int
    hkv: int
    d: int
    page: int = PAGE_SIZE
    scale: float | None = None  # defaults to fp32(1/sqrt(d))

    @property
    def softmax_scale(self) -> float:
        s = self.scale if self.scale is not None else 1.0 / math.sqrt(self.d)
        return float(np.float32(s))

    @property
    def group(self) -> int:
        return self.hq // self.hkv


@dataclasses.dataclass
class Batch:
    shape: Shape
    q_len: np.ndarray        # int32 [n]   c_i
    ctx_len: np.ndarray      # int32 [n]   u_i
    block_table: np.ndarray  # int32 [n, max_pages_per_req]
    num_pages: int
    q: np.ndarray            # uint16 [T, Hq, D]
    k_new: np.ndarray        # uint16 [T, Hkv, D]
    v_new: np.ndarray        # uint16 [T, Hkv, D]
    k_cache: np.ndarray      # uint16 [num_pages, Hkv, P, D]
    v_cache: np.ndarray      # uint16 [num_pages, Hkv, D, P]
    name: str = ""
    seed: int = 0

    @property
    def num_reqs(self) -> int:
        return int(self.q_len.shape[0])

    @property
    def num_tokens(self) -> int:
        return int(self.q_len.sum())

    @property
    def max_pages_per_req(self) -> int:
        return int(self.block_table.shape[1])

    def digest(self) -> str:
        h = hashlib.sha256()
        for a in (self.q_len, self.ctx_len, self.block_table, self.q, self.k_new,
                  self.v_new, self.k_cache, self.v_cache):
            h.update(np.ascontiguousarray(a).tobytes())
        return h.hexdigest()


_SLAB = 1 << 22


def _normal_bf16(rng: np.random.Generator, shape, std: float = 1.0) -> np.ndarray:
    """bf16 bits of fp32 N(0, std^2) draws.  Slab k of 2^22 values comes from its
    own PCG64 stream (spawned from ``rng``), so the result does not depend on how
    many threads fill the slabs."""
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.uint16)
    nslab = (n + _SLAB - 1) // _SLAB
    seeds = rng.bit_generator.seed_seq.spawn(nslab) if nslab else []

    def fill(k):
        s, e = k * _SLAB, min(n, (k + 1) * _SLAB)
        g = np.random.Generator(np.random.PCG64(seeds[k]))
        z = g.standard_normal(e - s, dtype=np.float32)
        if std != 1.0:
            z *= np.float32(std)
        out[s:e] = f32_to_bf16_bits(z)

    if nslab > 1:
        workers = max(1, min(16, len(os.sched_getaffinity(0))))
        with concurrent.futures.ThreadPoolExecutor(workers) as ex:
            list(ex.map(fill, range(nslab)))
    elif nslab == 1:
        fill(0)
    return out.reshape(shape)


def normal_bf16(shape, seed: int, std: float = 1.0) -> np.ndarray:
    """bf16 bits of seeded N(0, std^2) draws (activations, weights of the layer
    around attention)."""
    return _normal_bf16(np.random.default_rng(seed), tuple(shape), std)


def layer_weights(seed: int, hidden: int, inter: int, hq: int, hkv: int, d: int) -> dict:
    """Random weights of one Llama-style decoder layer, as bf16 bits in the
    torch Linear layout [out, in]: projections N(0, 1/fan_in), RMSNorm weights
    N(1, 0.1^2)."""
    shapes = {"w_q": (hq * d, hidden), "w_k": (hkv * d, hidden), "w_v": (hkv * d, hidden),
              "w_o": (hidden, hq * d), "w_gate": (inter, hidden), "w_up": (inter, hidden),
              "w_down": (hidden, inter)}
    out = {}
    for i, (name, shp) in enumerate(shapes.items()):
        out[name] = normal_bf16(shp, seed * 16 + i, shp[1] ** -0.5)
    for j, name in enumerate(("attn_norm", "mlp_norm")):
        z = np.random.default_rng(seed * 16 + 8 + j).standard_normal(hidden, dtype=np.float32)
        out[name] = f32_to_bf16_bits(np.float32(1.0) + np.float32(0.1) * z)
    return out


def make_batch(shape: Shape, q_len, ctx_len, seed: int = 0, spare_pages: int = 64,
               poison: bool = True, extra_pages_per_req: int = 0, name: str = "") -> Batch:
    """Draw a batch for the given per-request (c_i, u_i) lists."""
    q_len = np.asarray(q_len, dtype=np.int32).reshape(-1)
    ctx_len = np.asarray(ctx_len, dtype=np.int32).reshape(-1)
    if q_len.shape != ctx_len.shape:
        raise ValueError("q_len and ctx_len differ in length")
    if (q_len < 0).any() or (ctx_len < 0).any():
        raise ValueError("negative length")
    P = shape.page
    n = q_len.shape[0]
    T = int(q_len.sum())
    need = (ctx_len.astype(np.int64) + q_len + P - 1) // P
    total = int(need.sum())
    num_pages = total + int(spare_pages)
    maxp = int(need.max()) if n else 0
    maxp = max(1, maxp + int(extra_pages_per_req))

    ss = np.random.SeedSequence(seed)
    r_table, r_pool, r_new = (np.random.Generator(np.random.PCG64(s)) for s in ss.spawn(3))

    perm = r_table.permutation(num_pages).astype(np.int32)
    bt = np.full((n, maxp), -1, dtype=np.int32)
    off = 0
    for i in range(n):
        bt[i, : need[i]] = perm[off: off + need[i]]
        off += int(need[i])

    kc = _normal_bf16(r_pool, (num_pages, shape.hkv, P, shape.d))
    vc = _normal_bf16(r_pool, (num_pages, shape.hkv, shape.d, P))
    q = _normal_bf16(r_new, (T, shape.hq, shape.d))
    kn = _normal_bf16(r_new, (T, shape.hkv, shape.d))
    vn = _normal_bf16(r_new, (T, shape.hkv, shape.d))

    fill = BF16_NAN if poison else np.uint16(0)
    used = np.zeros(num_pages, dtype=bool)
    for i in range(n):
        pages = bt[i, : need[i]]
        used[pages] = True
        u = int(ctx_len[i])
        # positions >= u of this request are not cached yet: slots the append fills
        # and the unused tail of the last page.
        for lp in range(u // P, int(need[i])):
            s0 = max(0, u - lp * P)
            kc[pages[lp], :, s0:, :] = fill
            vc[pages[lp], :, :, s0:] = fill
    kc[~used] = fill
    vc[~used] = fill
    return Batch(shape, q_len, ctx_len, bt, num_pages, q, kn, vn, kc, vc, name=name, seed=seed)


# ---------------------------------------------------------------------------
# Workloads shaped like the paper's evaluation (Sec. 5: Llama3-8B / Qwen2.5-7B
# class attention shapes; Tab. 2 prompt lengths), at one GPU's full head count.
# ---------------------------------------------------------------------------

def _lognormal_int(rng, mu, sigma, lo, hi, n):
    x = np.rint(rng.lognormal(mean=mu, sigma=sigma, size=n))
    return np.clip(x, lo, hi).astype(np.int32)


def workload_lengths(name: str, seed: int = 0, chunk: int | None = None,
                     prefix: int | None = None):
    """(Shape, q_len, ctx_len) of a named workload.

    Names:
      tiny        8q/8kv/D64: 1 chunk (u=192, c=64) + decodes u in {128,256,384,512}
      l8b         32q/8kv/D128: 1 chunk (u=2048, c=512) + 64 decodes, u ~ U[512,4096]
      l8b_sweep   32q/8kv/D128: 1 chunk of an 8192-token prompt at prefix in
                  {0,2048,6144}, c in {128..2048} + 128 decodes, u ~ round(LogN(7.0,0.8))
                  clipped to [64,8192]
      multi       28q/4kv/D128: 4 chunks c in {64,256,512,1024}, u ~ U[0,8192]
                  + 256 decodes, u ~ round(LogN(7.2,1.0)) clipped to [64,16384]
      l70b        64q/8kv/D128: 1 chunk (u=32768, c=1024) + 32 decodes, u ~ U[8192,32768]
      l70b_tp8    one GPU's share of l70b under 8-way head parallelism: 8q/1kv/D128,
                  the same lengths
    ``chunk`` / ``prefix`` override the chunk size / prefix of the first chunk
    request (the chunk-size sweep knob); ``chunk=0`` leaves a pure-decode batch.
    Uniform integers are inclusive at both ends; lognormal draws are rounded then
    clipped.
    """
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 7])))
    if name == "tiny":
        shape = Shape(8, 8, 64)
        c = [64 if chunk is None else chunk] + [1] * 4
        u = [192 if prefix is None else prefix, 128, 256, 384, 512]
    elif name == "l8b":
        shape = Shape(32, 8, 128)
        dec = rng.integers(512, 4096, size=64, endpoint=True)
        c = [512 if chunk is None else chunk] + [1] * 64
        u = [2048 if prefix is None else prefix] + dec.tolist()
    elif name == "l8b_sweep":
        shape = Shape(32, 8, 128)
        dec = _lognormal_int(rng, 7.0, 0.8, 64, 8192, 128)
        c = [512 if chunk is None else chunk] + [1] * 128
        u = [2048 if prefix is None else prefix] + dec.tolist()
    elif name == "multi":
        shape = Shape(28, 4, 128)
        pre = rng.integers(0, 8192, size=4, endpoint=True)
        dec = _lognormal_int(rng, 7.2, 1.0, 64, 16384, 256)
        chunks = [64, 256, 512, 1024]
        if chunk is not None:  # scale the four chunks by chunk/512
            chunks = [max(0, int(round(x * chunk / 512))) for x in chunks]
        c = chunks + [1] * 256
        u = pre.tolist() + dec.tolist()
    elif name in ("l70b", "l70b_tp8"):
        shape = Shape(64, 8, 128) if name == "l70b" else Shape(8, 1, 128)
        dec = rng.integers(8192, 32768, size=32, endpoint=True)
        c = [1024 if chunk is None else chunk] + [1] * 32
        u = [32768 if prefix is None else prefix] + dec.tolist()
    else:
        raise KeyError(name)
    q_len = np.asarray(c, dtype=np.int32)
    ctx_len = np.asarray(u, dtype=np.int32)
    if chunk == 0:  # pure decode scene: drop the zero-token chunk requests
        keep = q_len > 0
        q_len, ctx_len = q_len[keep], ctx_len[keep]
    return shape, q_len, ctx_len


WORKLOADS = ("tiny", "l8b", "l8b_sweep", "multi", "l70b", "l70b_tp8")


def make_workload(name: str, seed: int = 0, chunk: int | None = None,
                  prefix: int | None = None, poison: bool = True) -> Batch:
    shape, q_len, ctx_len = workload_lengths(name, seed, chunk, prefix)
    return make_batch(shape, q_len, ctx_len, seed=seed, poison=poison, name=name)


def sub_batch(b: Batch, keep) -> Batch:
    """The batch restricted to the requests in ``keep`` (bool mask or indices),
    sharing the same pools: used for the pure-decode / pure-prefill scenes."""
    idx = np.arange(b.num_reqs)[keep] if np.asarray(keep).dtype == bool else np.asarray(keep)
    starts = np.concatenate([[0], np.cumsum(b.q_len)]).astype(np.int64)
    rows = np.concatenate([np.arange(starts[i], starts[i + 1]) for i in idx]) if len(idx) else np.zeros(0, np.int64)
    return Batch(b.shape, b.q_len[idx].copy(), b.ctx_len[idx].copy(), b.block_table[idx].copy(),
                 b.num_pages, b.q[rows], b.k_new[rows], b.v_new[rows], b.k_cache, b.v_cache,
                 name=b.name, seed=b.seed)
