"""ssa_append_attention_streams on an MI355X, through the C ABI: the chunk rows
on one stream and the decode rows (their own kernel, built to run beside the
chunk tiles) on a second one.

Against the fp64 oracle: the pool image bit for bit (NaN-poisoned new slots and
spare bytes), every output within the attention bars, the status word and the
launch counters at zero.  Against the one-launch path with the same plan: the
chunk rows' outputs bit for bit (the same kernel code), the decode rows within
the bars of the oracle (their kernel sums over the head dim in another order).
"""
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

MAX_ABS = 2e-2
MEAN_ABS = 2e-3


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def torch_dev():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    torch.cuda.set_device(0)
    return torch


def assert_close(got, ref, what=""):
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    err = np.abs(got.astype(np.float64) - ref)
    say(f"    {what}: max_abs={err.max() if err.size else 0:.3e} "
        f"mean_abs={err.mean() if err.size else 0:.3e} n={err.size}")
    if err.size:
        assert err.max() <= MAX_ABS, f"{what}: max abs {err.max()}"
        assert err.mean() <= MEAN_ABS, f"{what}: mean abs {err.mean()}"


def tuning(**kw):
    """The split forced (mix_order 6): chunk items first, half of the decode
    items beside the chunk rows and half after them, whatever the batch."""
    from paper_2606_05933_amd import ssa
    return ssa.make_tuning(mix_order=6, **kw)


def streams_parity(b, tu=None, plan_on_device=False, ref=None):
    """Both paths on fresh (poisoned) pools from one oracle evaluation."""
    import torch
    from oracle import oracle
    from paper_2606_05933_amd.device import DeviceBatch, bits_of
    tu = tu or tuning()
    if ref is None:
        kc, vc = oracle.batch_kv_append(b)
        out_ref, _ = oracle.batch_attention(b, kc, vc)
    else:
        kc, vc, out_ref = ref
    say(f"[gpu streams] {b.name} reqs={b.num_reqs} T={b.num_tokens} hq/hkv/d={b.shape.hq}/"
        f"{b.shape.hkv}/{b.shape.d} seed={b.seed}")
    db = DeviceBatch(b, tu, plan_on_device=plan_on_device)
    db.step_streams()
    torch.cuda.synchronize()
    assert np.array_equal(bits_of(db.k_cache).reshape(kc.shape), kc), "K pool image differs"
    assert np.array_equal(bits_of(db.v_cache).reshape(vc.shape), vc), "V pool image differs"
    assert_close(db.out_f32(), out_ref, b.name + " streams")
    assert db.status() == 0, f"status word {db.status()}"
    assert not db.launch_words().any()
    one = DeviceBatch(b, tu, plan_on_device=plan_on_device)
    one.step_fused()
    torch.cuda.synchronize()
    chunk_rows = torch.from_numpy(np.repeat(b.q_len > 1, b.q_len)).to(db.out.device)
    got, want = db.out[chunk_rows], one.out[chunk_rows]
    assert torch.equal(got.view(torch.int16), want.view(torch.int16)), "chunk rows differ"
    return db


def small(hq, hkv, d, cu, seed=0, name="small"):
    from paper_2606_05933_amd import workload
    return workload.make_batch(workload.Shape(hq, hkv, d), [c for c, _ in cu], [u for _, u in cu],
                               seed=seed, spare_pages=7, name=name)


SMALL = [
    # the decode kernel: G = 1, 4, 7, 8 at D = 128; lengths around the block,
    # page and piece boundaries; c = 0 rows; decode rows only
    (32, 8, 128, [(1, 0), (1, 1), (1, 15), (1, 16), (1, 31), (1, 32), (1, 33), (0, 7)]),
    (32, 8, 128, [(17, 0), (1, 0), (33, 31), (0, 0), (1, 47), (1, 3071), (1, 3072), (1, 3073)]),
    (28, 4, 128, [(64, 0), (1, 100), (100, 1000), (1, 2047)]),        # G = 7
    (64, 8, 128, [(70, 400), (1, 1), (1, 4097), (1, 20000)]),        # G = 8
    (4, 4, 128, [(300, 77), (1, 129)]),                               # G = 1
    (32, 8, 128, [(1, 65535), (1, 12287), (40, 20000)]),              # many decode pieces
    # the one-launch fallback: D = 64, G = 16
    (8, 8, 64, [(1, 0), (0, 5), (2, 0), (1, 15), (1, 16), (1, 31), (1, 32), (1, 33)]),
    (64, 4, 128, [(129, 0), (1, 0), (3, 700)]),
]


@pytest.mark.parametrize("case", range(len(SMALL)))
def test_streams_small_batches(torch_dev, case):
    hq, hkv, d, cu = SMALL[case]
    streams_parity(small(hq, hkv, d, cu, seed=case, name=f"streams{case}"))


@pytest.mark.parametrize("name", ["tiny", "l8b", "multi", "l70b_tp8"])
def test_streams_workloads(torch_dev, name):
    from paper_2606_05933_amd import workload
    streams_parity(workload.make_workload(name, seed=1))


def test_streams_full_size_l70b(torch_dev):
    """The 70B-shaped mixed batch at full size, every element."""
    from paper_2606_05933_amd import workload
    streams_parity(workload.make_workload("l70b", seed=0))


def test_streams_with_splits_and_device_plan(torch_dev):
    b = small(32, 8, 128, [(300, 1500), (1, 3000), (1, 5000), (64, 0), (1, 777)], seed=5,
              name="streams-split")
    streams_parity(b, tuning(chunk_split_keys=512, decode_split_keys=1024), plan_on_device=True)


def test_streams_repeated_from_poisoned_pools(torch_dev):
    """Every call starts from pools with the new slots NaN-poisoned (a read of a
    new row before its append shows); all calls give the same bytes, and the
    counters and merge tickets end at zero."""
    import torch
    from paper_2606_05933_amd import workload
    from paper_2606_05933_amd.device import DeviceBatch
    b = workload.make_workload("multi", seed=6)
    db = DeviceBatch(b, tuning(decode_split_keys=1024))
    k0, v0 = db.k_cache.clone(), db.v_cache.clone()
    db.step_streams()
    torch.cuda.synchronize()
    ref = db.out.clone()
    for k in range(20):
        db.k_cache.copy_(k0)
        db.v_cache.copy_(v0)
        db.out.zero_()
        db.replan_host()
        db.step_streams()
        torch.cuda.synchronize()
        assert torch.equal(db.out.view(torch.int16), ref.view(torch.int16)), k
    assert db.status() == 0 and not db.launch_words().any()


def test_streams_automatic_split_on_the_70b_batch_and_one_launch_elsewhere(torch_dev):
    """mix_order 5: the 70B-shaped batch splits (every decode item beside the
    chunk rows) and matches the oracle; the 8B-shaped batch keeps one launch,
    bit for bit the fused call with the same plan."""
    import torch
    from paper_2606_05933_amd import ssa, workload
    from paper_2606_05933_amd.device import DeviceBatch
    b = workload.make_workload("l70b", seed=2)
    db = streams_parity(b, ssa.make_tuning(mix_order=5))
    assert db.plan_header_field("streams_beside") == db.info.num_decode_items
    b = workload.make_workload("l8b", seed=2)
    s = DeviceBatch(b, ssa.make_tuning(mix_order=5))
    assert s.plan_header_field("streams_beside") == -1
    f = DeviceBatch(b, ssa.make_tuning(mix_order=5))
    s.step_streams()
    f.step_fused()
    torch.cuda.synchronize()
    assert torch.equal(s.out.view(torch.int16), f.out.view(torch.int16))
    assert s.status() == 0 and not s.launch_words().any()


def test_streams_plan_without_split_runs_as_one_launch(torch_dev):
    """A plan of another order (here interleaved) runs as one launch on the
    launch stream: bit for bit ssa_append_attention with the same plan."""
    import torch
    from paper_2606_05933_amd import ssa, workload
    from paper_2606_05933_amd.device import DeviceBatch
    b = workload.make_workload("multi", seed=4)
    s = DeviceBatch(b, ssa.make_tuning(mix_order=2))
    f = DeviceBatch(b, ssa.make_tuning(mix_order=2))
    assert s.plan_header_field("streams_beside") == -1
    s.step_streams()
    f.step_fused()
    torch.cuda.synchronize()
    assert torch.equal(s.out.view(torch.int16), f.out.view(torch.int16))
    assert torch.equal(s.k_cache.view(torch.int16), f.k_cache.view(torch.int16))


def test_streams_events_stamp_the_chunk_launch(torch_dev):
    """Timing events are stamped by the chunk rows' launch itself (the pair's
    longest kernel): inside the span of events recorded on the stream around
    the call; timed calls give the same bytes as untimed ones."""
    import torch
    from paper_2606_05933_amd import workload
    from paper_2606_05933_amd.device import DeviceBatch
    b = workload.make_workload("l8b", seed=3)
    db = DeviceBatch(b, tuning())
    db.step_streams()
    torch.cuda.synchronize()
    ref = db.out.clone()
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    for e in evs:
        e.record()
    db.out.zero_()
    torch.cuda.synchronize()
    outer0, k0, k1, outer1 = evs
    outer0.record()
    db.step_streams(events=(k0, k1))
    outer1.record()
    torch.cuda.synchronize()
    assert torch.equal(db.out.view(torch.int16), ref.view(torch.int16))
    kernel_us, span_us = k0.elapsed_time(k1) * 1e3, outer0.elapsed_time(outer1) * 1e3
    say(f"    chunk launch {kernel_us:.1f} us, whole call {span_us:.1f} us")
    assert 0 < kernel_us <= span_us
    assert outer0.elapsed_time(k0) >= 0 and k1.elapsed_time(outer1) >= 0


def test_streams_call_replays_from_a_graph(torch_dev):
    """The fork/join of the two streams captured in a HIP graph (the decode
    stream joins the capture through the fork event) and replayed, with eager
    work and synchronisations between replays: every replay gives the eager
    call's bytes.  The library's events are created by an eager call first."""
    import torch
    from paper_2606_05933_amd import workload
    from paper_2606_05933_amd.device import DeviceBatch
    b = small(32, 8, 128, [(300, 1500), (1, 3000), (1, 5000), (64, 0), (1, 9000)], seed=11,
              name="streams-graph")
    db = DeviceBatch(b, tuning())
    k0, v0 = db.k_cache.clone(), db.v_cache.clone()
    db.step_streams()
    torch.cuda.synchronize()
    ref, kref, vref = db.out.clone(), db.k_cache.clone(), db.v_cache.clone()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        call = __import__("paper_2606_05933_amd.ssa", fromlist=["ssa"]).bind_append_attention_streams(
            db.shape, db.plan_host, db.plan_dev, db.q, db.k_new, db.v_new, db.k_cache, db.v_cache,
            db.block_table, db.out, db.workspace, decode_stream=db.decode_stream)
        with torch.cuda.graph(g, stream=side):
            call()
    torch.cuda.synchronize()
    junk = torch.empty(1 << 20, dtype=torch.float32, device="cuda")
    for r in range(4):
        db.k_cache.copy_(k0)
        db.v_cache.copy_(v0)
        db.out.fill_(0)
        junk.uniform_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        say(f"    replay {r}")
        assert torch.equal(db.out.view(torch.int16), ref.view(torch.int16)), f"replay {r}"
        assert torch.equal(db.k_cache.view(torch.int16), kref.view(torch.int16))
        assert torch.equal(db.v_cache.view(torch.int16), vref.view(torch.int16))
    assert db.status() == 0 and not db.launch_words().any()
