"""A batch resident in device memory, with its plan, output and workspace.

Marshalling around the C ABI for tests, the benchmark and the smoke check:
uploads the arrays of a generated batch once, plans on the host into pinned,
device-mapped buffers that the kernels read in place (or, optionally, copies
the plan to device memory), and calls ``ssa_kv_append`` and
``ssa_mixed_attention`` on the current stream.
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


class DeviceBatch:
    def __init__(self, b, tuning: ssa.SsaTuning | None = None, device="cuda",
                 plan_on_device=False, pools=None):
        """plan_on_device: False, the kernels read the plan in place from pinned,
        device-mapped host memory; True, each re-plan is copied to device memory
        on the launch stream; "async", copied on a side stream that the launch
        stream waits for (the copy overlaps the previous iteration's kernels).
        pools: optional (k_cache, v_cache, block_table) device tensors of another
        DeviceBatch over the same pools, used instead of uploading b's."""
        if plan_on_device not in (False, True, "async"):
            raise ValueError("plan_on_device: False, True or 'async'")
        self.b = b
        self.plan_on_device = plan_on_device
        self.device = torch.device(device)
        s = b.shape
        self.shape = ssa.make_shape(s.hq, s.hkv, s.d, b.num_pages, b.max_pages_per_req,
                                    s.softmax_scale, s.page)
        self.tuning = tuning
        dev = self.device
        self.q = bf16_tensor(b.q, dev)
        self.k_new = bf16_tensor(b.k_new, dev)
        self.v_new = bf16_tensor(b.v_new, dev)
        if pools is not None:
            self.k_cache, self.v_cache, self.block_table = pools
        else:
            self.k_cache = bf16_tensor(b.k_cache, dev)
            self.v_cache = bf16_tensor(b.v_cache, dev)
            self.block_table = torch.from_numpy(np.ascontiguousarray(b.block_table)).to(dev)
        self.out = torch.zeros((b.num_tokens, s.hq, s.d), dtype=torch.bfloat16, device=dev)
        self.plan()

    def plan(self, tuning: ssa.SsaTuning | None = None):
        """(Re)build the plan on the host.

        Two plan slots alternate between iterations.  Each is a pinned,
        device-mapped host buffer that the kernels read directly (no copy), or,
        with ``plan_on_device``, a pinned buffer plus a device copy."""
        if tuning is not None:
            self.tuning = tuning
        b = self.b
        torch.cuda.synchronize(self.device)
        nbytes, ws_bytes = ssa.ssa_plan_size(self.shape, b.q_len, b.ctx_len, self.tuning)
        nbytes = max(nbytes, 128)
        self._host = [torch.zeros(nbytes, dtype=torch.uint8).pin_memory() for _ in range(2)]
        if self.plan_on_device:
            self._dev = [torch.empty(nbytes, dtype=torch.uint8, device=self.device)
                         for _ in range(2)]
        else:
            self._dev = self._host  # device-mapped pinned memory, read in place
        # the stream the calls are bound to, and (async copies) the side stream
        self._stream = torch.cuda.current_stream(self.device)
        if self.plan_on_device == "async":
            self._copy_stream = torch.cuda.Stream(self.device)
            self._copied = [torch.cuda.Event(), torch.cuda.Event()]
        # "the slot's kernels are done": the attention launch of the slot stamps
        # its own end into one of these (no extra packet on the stream)
        self._own_done = [torch.cuda.Event(), torch.cuda.Event()]
        for ev in self._own_done:
            ev.record()  # creates the HIP event
        self._done = list(self._own_done)
        self._used = [False, False]
        self._slot = 0
        _, self.info = ssa.ssa_plan(self.shape, b.q_len, b.ctx_len, self.tuning,
                                    out=self._host[0])
        # every entry the kernels will read names a real page (ssa_check_block_table)
        ssa.check_block_table(self.shape, self._host[0], b.block_table)
        if self.plan_on_device:
            self._dev[0].copy_(self._host[0])
        self.plan_host, self.plan_dev = self._host[0], self._dev[0]
        if not hasattr(self, "workspace") or self.workspace.numel() < ws_bytes:
            self.workspace = torch.zeros(max(ws_bytes, 256), dtype=torch.uint8, device=self.device)
        else:
            # another plan's split records may lie where this plan's tickets are
            self.workspace.zero_()
        # calls bound once per slot (on the stream current now): an iteration
        # only crosses into the library
        self._info_scratch = ssa.SsaPlanInfo()
        if not hasattr(self, "decode_stream"):
            # the second stream of ssa_append_attention_streams
            self.decode_stream = torch.cuda.Stream(self.device)
        self._bound = []
        for hb, db in zip(self._host, self._dev):
            self._bound.append((
                ssa.bind_plan(self.shape, b.q_len, b.ctx_len, self.tuning, hb, self._info_scratch),
                ssa.bind_kv_append(self.shape, hb, db, self.k_new, self.v_new, self.k_cache,
                                   self.v_cache, self.block_table),
                ssa.bind_mixed_attention(self.shape, hb, db, self.q, self.k_cache, self.v_cache,
                                         self.block_table, self.out, self.workspace),
                ssa.bind_append_attention(self.shape, hb, db, self.q, self.k_new, self.v_new,
                                          self.k_cache, self.v_cache, self.block_table, self.out,
                                          self.workspace),
                ssa.bind_append_attention_streams(self.shape, hb, db, self.q, self.k_new,
                                                  self.v_new, self.k_cache, self.v_cache,
                                                  self.block_table, self.out, self.workspace,
                                                  decode_stream=self.decode_stream)))
        torch.cuda.synchronize(self.device)
        return self.info

    def replan_host(self):
        """Plan the (same) batch again on the host into the other slot, as a
        serving loop does every iteration: wait until the kernels that last read
        that slot have finished, plan into it, and (with plan_on_device) copy it
        to its device buffer, on the launch stream or (async) on a side stream
        the launch stream waits for."""
        slot = self._slot ^ 1
        if self._used[slot]:
            self._done[slot].synchronize()
        self._bound[slot][0]()
        if self.plan_on_device == "async":
            # the slot's last kernels have finished (waited for above), so its
            # device copy may be overwritten at once; the launch stream waits
            with torch.cuda.stream(self._copy_stream):
                self._dev[slot].copy_(self._host[slot], non_blocking=True)
            self._copied[slot].record(self._copy_stream)
            self._stream.wait_event(self._copied[slot])
        elif self.plan_on_device:
            self._dev[slot].copy_(self._host[slot], non_blocking=True)
        self._used[slot] = True
        self._slot = slot
        self.plan_host, self.plan_dev = self._host[slot], self._dev[slot]

    def kv_append(self, stream=None, events=(None, None)):
        """events: optional (start, stop) torch.cuda.Event pair stamped with the
        kernel's own start and end (current stream only)."""
        if stream is None:
            self._bound[self._slot][1](*events)
        else:
            ssa.ssa_kv_append(self.shape, self.plan_host, self.plan_dev, self.k_new, self.v_new,
                              self.k_cache, self.v_cache, self.block_table, stream)

    def attention(self, stream=None, events=(None, None)):
        """events: optional (start, stop) pair stamped by the kernel; the stop
        event then also marks the slot's kernels done."""
        if stream is None:
            start, stop = events
            if stop is None:
                stop = self._own_done[self._slot]
            self._bound[self._slot][2](start, stop)
            self._done[self._slot] = stop
        else:
            ssa.ssa_mixed_attention(self.shape, self.plan_host, self.plan_dev, self.q,
                                    self.k_cache, self.v_cache, self.block_table, self.out,
                                    self.workspace, stream)

    def step(self, stream=None):
        self.kv_append(stream)
        self.attention(stream)

    def step_fused(self, events=(None, None)):
        """kv_append and attention in one launch (ssa_append_attention) on the
        current stream; its stop event marks the slot's kernels done."""
        start, stop = events
        if stop is None:
            stop = self._own_done[self._slot]
        self._bound[self._slot][3](start, stop)
        self._done[self._slot] = stop

    def step_streams(self, events=(None, None)):
        """The iteration as two launches side by side (ssa_append_attention_streams):
        the chunk rows on the current stream, the decode rows on this batch's
        decode stream, joined back into the current stream, where the plan asks
        for it (tuning mix_order 5 or 6); otherwise the one launch.  events:
        optional (start, stop) pair stamped by the chunk rows' launch."""
        self._bound[self._slot][4](*events)
        # the events (if any) stamp the chunk rows' launch only: the slot is done
        # once the launch stream has joined the decode stream, after the call
        done = self._own_done[self._slot]
        done.record()
        self._done[self._slot] = done

    def status(self) -> int:
        """The workspace's status word (ssa.h: SSA_STATUS_* bits) after the
        launches issued so far have completed."""
        torch.cuda.synchronize(self.device)
        o = ssa.SSA_WS_STATUS_OFFSET
        return int(self.workspace[o:o + 4].view(torch.int32).item())

    def clear_status(self):
        o = ssa.SSA_WS_STATUS_OFFSET
        self.workspace[o:o + 4].zero_()

    def launch_words(self) -> np.ndarray:
        """The fused launch's counters, the status word and the merge tickets
        (int32, host copy): every word but the status is zero at rest."""
        n = ssa.WS_LAUNCH_WORDS + self.info.num_merge_groups
        return self.workspace[:4 * n].view(torch.int32).cpu().numpy()

    def plan_header_field(self, name: str) -> int:
        """An int32 field of the current plan's header (ssa_plan_format.h)."""
        fields = {"num_items": 6, "num_chunk_items": 7, "num_decode_items": 8,
                  "wait_polls": 30, "streams_beside": 31}
        return int(self.plan_host[:128].view(torch.int32)[fields[name]].item())

    def out_f32(self) -> np.ndarray:
        return self.out.float().cpu().numpy()
