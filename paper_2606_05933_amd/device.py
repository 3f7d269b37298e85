"""A batch resident in device memory, with its plan, output and workspace.

Marshalling around the C ABI for tests, the benchmark and the smoke check:
uploads the arrays of a generated batch once, plans on the host, copies the
plan blob to the device through a pinned buffer, and calls ``ssa_kv_append``
and ``ssa_mixed_attention`` on the current stream.
"""
from __future__ import annotations

import numpy as np
import torch

from . import ssa


def bf16_tensor(bits: np.ndarray, device) -> torch.Tensor:
    """Device bf16 tensor holding the given uint16 bit patterns."""
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.to(device).view(torch.bfloat16)


def bits_of(t: torch.Tensor) -> np.ndarray:
    """uint16 bit patterns of a bf16 tensor (copied to the host)."""
    return t.detach().view(torch.int16).cpu().numpy().view(np.uint16)


def check_block_table(block_table: np.ndarray, q_len, ctx_len, num_pages: int, page: int = 16):
    """Host-side check that every entry the kernels may read names a real page."""
    for i, (c, u) in enumerate(zip(q_len, ctx_len)):
        n = (int(u) + int(c) + page - 1) // page
        row = block_table[i, :n]
        if n > block_table.shape[1] or (row < 0).any() or (row >= num_pages).any():
            raise ValueError(f"block table row {i} names a page outside [0, {num_pages})")


class DeviceBatch:
    def __init__(self, b, tuning: ssa.SsaTuning | None = None, device="cuda"):
        self.b = b
        self.device = torch.device(device)
        s = b.shape
        check_block_table(b.block_table, b.q_len, b.ctx_len, b.num_pages, s.page)
        self.shape = ssa.make_shape(s.hq, s.hkv, s.d, b.num_pages, b.max_pages_per_req,
                                    s.softmax_scale, s.page)
        self.tuning = tuning
        dev = self.device
        self.q = bf16_tensor(b.q, dev)
        self.k_new = bf16_tensor(b.k_new, dev)
        self.v_new = bf16_tensor(b.v_new, dev)
        self.k_cache = bf16_tensor(b.k_cache, dev)
        self.v_cache = bf16_tensor(b.v_cache, dev)
        self.block_table = torch.from_numpy(np.ascontiguousarray(b.block_table)).to(dev)
        self.out = torch.zeros((b.num_tokens, s.hq, s.d), dtype=torch.bfloat16, device=dev)
        self.plan()

    def plan(self, tuning: ssa.SsaTuning | None = None):
        """(Re)build the plan on the host and copy it to the device."""
        if tuning is not None:
            self.tuning = tuning
        b = self.b
        nbytes, ws_bytes = ssa.ssa_plan_size(self.shape, b.q_len, b.ctx_len, self.tuning)
        # two pinned host buffers: the host plans into one while the copy out of
        # the other may still be queued on the stream
        self._ring = [torch.zeros(max(nbytes, 128), dtype=torch.uint8).pin_memory()
                      for _ in range(2)]
        self._ring_ev = [None, None]
        self._slot = 0
        self.plan_host = self._ring[0]
        _, self.info = ssa.ssa_plan(self.shape, b.q_len, b.ctx_len, self.tuning,
                                    out=self.plan_host)
        self.plan_dev = torch.empty_like(self.plan_host, device=self.device)
        self.plan_dev.copy_(self.plan_host, non_blocking=True)
        self._ring_ev[0] = torch.cuda.Event()
        self._ring_ev[0].record()
        if not hasattr(self, "workspace") or self.workspace.numel() < ws_bytes:
            self.workspace = torch.zeros(max(ws_bytes, 256), dtype=torch.uint8, device=self.device)
        return self.info

    def replan_host(self):
        """Host planning of the same batch into a pinned buffer (what a serving
        loop does every iteration), followed by the async copy to the device."""
        self._slot ^= 1
        buf, ev = self._ring[self._slot], self._ring_ev[self._slot]
        if ev is not None:
            ev.synchronize()  # the copy that last read this buffer has run
        ssa.ssa_plan(self.shape, self.b.q_len, self.b.ctx_len, self.tuning, out=buf)
        self.plan_host = buf
        self.plan_dev.copy_(buf, non_blocking=True)
        if ev is None:
            ev = self._ring_ev[self._slot] = torch.cuda.Event()
        ev.record()

    def kv_append(self, stream=None):
        ssa.ssa_kv_append(self.shape, self.plan_host, self.plan_dev, self.k_new, self.v_new,
                          self.k_cache, self.v_cache, self.block_table, stream)

    def attention(self, stream=None):
        ssa.ssa_mixed_attention(self.shape, self.plan_host, self.plan_dev, self.q, self.k_cache,
                                self.v_cache, self.block_table, self.out, self.workspace, stream)

    def step(self, stream=None):
        self.kv_append(stream)
        self.attention(stream)

    def out_f32(self) -> np.ndarray:
        return self.out.float().cpu().numpy()
