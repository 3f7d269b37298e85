"""Parity of the HIP path with the CPU oracle, through the C ABI, on an MI355X.

Bars: kv_append bit-exact (the whole pool image, untouched bytes included);
attention within max |err| <= 2e-2 and mean |err| <= 2e-3 of the fp64 oracle on
bf16 outputs (fp32 accumulation on the GPU).  Pools are NaN-poisoned wherever a
kernel must not read (unwritten slots, the tail of a request's last page, spare
pages), so a leak shows up as a non-finite output.
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


def run(b, tuning=None, plan_on_device=False):
    import torch
    from paper_2606_05933_amd.device import DeviceBatch
    say(f"[gpu] {b.name} reqs={b.num_reqs} T={b.num_tokens} hq/hkv/d={b.shape.hq}/{b.shape.hkv}/"
        f"{b.shape.d} seed={b.seed} plan_on_device={plan_on_device}")
    db = DeviceBatch(b, tuning, plan_on_device=plan_on_device)
    db.step()
    torch.cuda.synchronize()
    return db


def assert_close(got, ref, what=""):
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    err = np.abs(got.astype(np.float64) - ref)
    say(f"    {what}: max_abs={err.max() if err.size else 0:.3e} "
        f"mean_abs={err.mean() if err.size else 0:.3e} n={err.size}")
    if err.size:
        assert err.max() <= MAX_ABS, f"{what}: max abs {err.max()}"
        assert err.mean() <= MEAN_ABS, f"{what}: mean abs {err.mean()}"


def full_parity(b, tuning=None, plan_on_device=False):
    from oracle import oracle
    from paper_2606_05933_amd.device import bits_of
    db = run(b, tuning, plan_on_device)
    kc, vc = oracle.batch_kv_append(b)
    assert np.array_equal(bits_of(db.k_cache).reshape(kc.shape), kc), "K pool image differs"
    assert np.array_equal(bits_of(db.v_cache).reshape(vc.shape), vc), "V pool image differs"
    ref, _ = oracle.batch_attention(b, kc, vc)
    assert_close(db.out_f32(), ref, b.name)
    assert db.status() == 0, f"status word {db.status()}"
    return db


def small(hq, hkv, d, cu, seed=0, name="small"):
    from paper_2606_05933_amd import workload
    shape = workload.Shape(hq, hkv, d)
    q_len = [c for c, _ in cu]
    ctx = [u for _, u in cu]
    return workload.make_batch(shape, q_len, ctx, seed=seed, spare_pages=7, name=name)


SMALL = [
    # edge cases: u = 0, a single key, c = 0 rows, unaligned prefixes, chunks crossing pages
    (8, 8, 64, [(1, 0)]),
    (8, 8, 64, [(1, 0), (0, 5), (2, 0), (1, 15), (1, 16), (1, 31), (1, 32), (1, 33)]),
    (32, 8, 128, [(17, 0), (1, 0), (33, 31), (0, 0), (1, 47)]),
    (28, 4, 128, [(64, 0), (1, 100), (100, 1000), (1, 2047)]),        # G = 7
    (64, 8, 128, [(70, 400), (1, 1), (1, 4097)]),                    # G = 8
    (16, 1, 64, [(40, 60), (1, 500)]),                               # G = 16
    (4, 4, 128, [(300, 77), (1, 129)]),                               # G = 1, D = 128
    (12, 4, 64, [(2, 0), (3, 1), (65, 1023), (1, 0)]),                # G = 3, D = 64
    (64, 4, 128, [(129, 0), (1, 0), (3, 700)]),                       # G = 16, D = 128
    (8, 8, 64, [(2048, 0), (1, 1)]),                                  # long chunk from empty
    (32, 8, 128, [(1, 65535), (1, 12287), (40, 20000)]),              # many decode pieces
]


def test_repeat_launches_are_bitwise_identical_and_reset_tickets(torch_dev):
    """1000 launches with merge groups: every output the same bytes, and the
    tickets back at zero after each (the last arriver of a group resets it)."""
    import torch
    from paper_2606_05933_amd import ssa
    b = small(32, 8, 128, [(300, 1500), (1, 3000), (1, 5000)], seed=3, name="repeat")
    db = run(b, ssa.make_tuning(chunk_split_keys=512, decode_split_keys=256))
    assert db.info.num_merge_groups > 0
    first = db.out.clone()
    for k in range(1000):
        db.out.zero_()
        db.attention()
        if k % 100 == 99:
            torch.cuda.synchronize()
            assert torch.equal(db.out.view(torch.int16), first.view(torch.int16)), k
            assert not db.launch_words().any(), k
    torch.cuda.synchronize()
    assert not db.launch_words().any()


@pytest.mark.parametrize("case", range(len(SMALL)))
def test_small_batches_match_oracle(torch_dev, case):
    hq, hkv, d, cu = SMALL[case]
    full_parity(small(hq, hkv, d, cu, seed=case, name=f"small{case}"))


def test_tiny_workload_matches_oracle(torch_dev):
    from paper_2606_05933_amd import workload
    full_parity(workload.make_workload("tiny", seed=0))


@pytest.mark.parametrize("plan_on_device", [False, True, "async"])
def test_llama8b_mixed_full_parity(torch_dev, plan_on_device):
    from paper_2606_05933_amd import workload
    full_parity(workload.make_workload("l8b", seed=0), plan_on_device=plan_on_device)


@pytest.mark.parametrize("plan_on_device", [False, "async"])
def test_replanned_iterations_alternate_plan_slots(torch_dev, plan_on_device):
    """Several iterations in a row, each re-planned into the other plan slot
    while the previous one may still run (with "async", each plan copied to the
    device on a side stream): every output matches the oracle."""
    import torch
    from oracle import oracle
    from paper_2606_05933_amd import workload
    from paper_2606_05933_amd.device import DeviceBatch
    b = workload.make_workload("l8b", seed=2)
    db = DeviceBatch(b, plan_on_device=plan_on_device)
    db.step()
    for k in range(6):
        db.replan_host()
        db.out.zero_()
        if k % 2:
            db.step_fused()
        else:
            db.step()
    torch.cuda.synchronize()
    assert db.status() == 0
    kc, vc = oracle.batch_kv_append(b)
    ref, _ = oracle.batch_attention(b, kc, vc)
    assert_close(db.out_f32(), ref, "l8b replanned")


@pytest.mark.parametrize("tile,csplit,dsplit", [(32, 0, 0), (64, 1024, 256), (128, 512, 128),
                                                (128, 0, 4096)])
def test_tuning_variants_match_oracle(torch_dev, tile, csplit, dsplit):
    from paper_2606_05933_amd import ssa
    b = small(32, 8, 128, [(300, 1500), (1, 3000), (1, 100), (45, 0)], seed=11, name="tuned")
    full_parity(b, ssa.make_tuning(chunk_tile_cols=tile, chunk_split_keys=csplit,
                                   decode_split_keys=dsplit))


def test_launch_orders_give_bitwise_identical_outputs(torch_dev):
    """The launch order only changes which workgroup runs when: every order
    gives the same bytes (splits merge in split order)."""
    import torch
    from paper_2606_05933_amd import ssa, workload
    b = workload.make_workload("multi", seed=4)
    db = run(b)
    ref = db.out.clone()
    for order in (2, 3, 4):
        for cus in (256, 7):
            db.plan(ssa.make_tuning(mix_order=order, num_cus=cus))
            db.out.zero_()
            db.attention()
            torch.cuda.synchronize()
            assert torch.equal(db.out.view(torch.int16), ref.view(torch.int16)), (order, cus)


def test_scenes_pure_decode_and_pure_prefill(torch_dev):
    from paper_2606_05933_amd import workload
    b = workload.make_workload("l8b", seed=1)
    dec = workload.sub_batch(b, b.q_len == 1)
    dec.name = "l8b-pure-decode"
    db = full_parity(dec)
    assert db.info.scene == 1
    pre = workload.sub_batch(b, b.q_len > 1)
    pre.name = "l8b-pure-prefill"
    db = full_parity(pre)
    assert db.info.scene == 2


def sampled_parity(b, n_chunk_rows=24, heads_per_row=4, seed=0):
    """Oracle at sampled (row, head) pairs of a full-size batch."""
    from oracle import oracle
    db = run(b)
    out = db.out_f32()
    rng = np.random.default_rng(seed)
    starts = np.concatenate([[0], np.cumsum(b.q_len)])
    rows = []
    for i in range(b.num_reqs):
        c = int(b.q_len[i])
        if c == 1:
            rows.append(starts[i])
        elif c > 1:
            pick = {0, 1, c - 1, c // 2} | set(rng.integers(0, c, size=n_chunk_rows).tolist())
            rows.extend(starts[i] + j for j in sorted(pick))
    sel_rows, sel_heads = [], []
    for r in rows:
        for h in rng.choice(b.shape.hq, size=min(heads_per_row, b.shape.hq), replace=False):
            sel_rows.append(r)
            sel_heads.append(h)
    s = b.shape
    # the device pools hold the appended rows; the oracle appends on its own copy
    kc, vc = oracle.batch_kv_append(b)
    ref, _ = oracle.attention_rows(s.hq, s.hkv, s.d, s.page, s.softmax_scale, b.q_len, b.ctx_len,
                                   b.block_table, b.q, kc, vc, np.array(sel_rows),
                                   np.array(sel_heads))
    got = out[np.array(sel_rows), np.array(sel_heads)]
    assert_close(got, ref, f"{b.name} sampled")
    assert np.isfinite(out).all(), "non-finite output outside the sample"
    assert db.status() == 0
    return db.out.clone()


@pytest.mark.parametrize("name,chunk,prefix", [
    ("multi", 1024, None), ("l70b", 2048, None), ("l8b", 2048, None), ("l70b", 1536, None),
    ("l70b_tp8", 2048, 131072), ("l70b_tp8", 4096, 262144),
])
def test_extra_sweep_rows_sampled_parity(torch_dev, name, chunk, prefix):
    """Latency-table rows beyond the five configurations (chunk sizes of the
    sweep; at c = 1536 the planner cuts every 70B chunk tile in two key pieces
    to fill the last round of workgroup slots), and long contexts (a chunk on a
    128K- or 256K-token prefix: chunk tiles of up to 266K keys cut into many
    key pieces): the oracle at sampled (row, head) pairs, and the fused launch
    equal to the two launches bit for bit."""
    import torch
    from paper_2606_05933_amd import workload
    from paper_2606_05933_amd.device import DeviceBatch
    b = workload.make_workload(name, seed=0, chunk=chunk, prefix=prefix)
    b.name = f"{name}(c={chunk},u={prefix})"
    two = sampled_parity(b)
    say(f"[gpu fused] {b.name}")
    fz = DeviceBatch(b)
    fz.step_fused()
    torch.cuda.synchronize()
    assert fz.status() == 0
    assert torch.equal(fz.out.view(torch.int16), two.view(torch.int16)), "fused != two launches"


def both_paths_parity(b):
    """One oracle evaluation, checked against both launch paths on fresh
    (poisoned) pools: ssa_kv_append + ssa_mixed_attention, and the fused
    ssa_append_attention.  Pool images bit for bit, every output element within
    the bars, the two paths' outputs identical bit for bit, status word zero."""
    import time
    import torch
    from oracle import oracle
    from paper_2606_05933_amd.device import DeviceBatch, bits_of
    t0 = time.time()
    kc, vc = oracle.batch_kv_append(b)
    ref, used = oracle.batch_attention(b, kc, vc)
    say(f"    oracle {time.time() - t0:.1f} s on {used} threads")
    outs = []
    for fused in (False, True):
        say(f"[gpu {'fused' if fused else 'two launches'}] {b.name} reqs={b.num_reqs} "
            f"T={b.num_tokens} hq/hkv/d={b.shape.hq}/{b.shape.hkv}/{b.shape.d} seed={b.seed}")
        db = DeviceBatch(b)
        if fused:
            db.step_fused()
        else:
            db.step()
        torch.cuda.synchronize()
        assert np.array_equal(bits_of(db.k_cache).reshape(kc.shape), kc), "K pool image differs"
        assert np.array_equal(bits_of(db.v_cache).reshape(vc.shape), vc), "V pool image differs"
        assert_close(db.out_f32(), ref, b.name + (" fused" if fused else ""))
        assert db.status() == 0 and not db.launch_words().any()
        outs.append(db.out.clone())
        del db
        torch.cuda.empty_cache()
    assert torch.equal(outs[0].view(torch.int16), outs[1].view(torch.int16)), "fused != two launches"


# Every element of every configuration at full size: the 15 (prefix, chunk) rows
# of the chunk-size sweep, the multi-chunk batch, the 70B-shaped layer and one
# GPU's share of it under 8-way head parallelism.
FULL_SIZE = ([("l8b_sweep", c, u) for u in (0, 2048, 6144) for c in (128, 256, 512, 1024, 2048)]
             + [("multi", None, None), ("l70b", None, None), ("l70b_tp8", None, None)])


@pytest.mark.parametrize("name,chunk,prefix", FULL_SIZE)
def test_full_size_parity_both_paths(torch_dev, name, chunk, prefix):
    from paper_2606_05933_amd import workload
    b = workload.make_workload(name, seed=0, chunk=chunk, prefix=prefix)
    b.name = f"{name}(c={chunk},u={prefix})"
    both_paths_parity(b)


def test_long_decode_contexts_both_paths(torch_dev):
    """Decode rows over 64K-256K cached tokens (up to 64 key pieces per row and
    kv head, merged in one group) beside a chunk on an empty cache: every
    element against the oracle on both launch paths."""
    from paper_2606_05933_amd import workload
    b = workload.make_batch(workload.Shape(16, 2, 128), [1, 1, 1, 1, 256],
                            [262143, 200000, 131071, 65536, 0], seed=7, spare_pages=3,
                            name="long-decodes")
    both_paths_parity(b)


def test_random_small_batches_both_paths(torch_dev):
    """100 seeded random batches: group size 1..16, head dim 64 or 128, 1..6
    requests with c in [0, 300] (a third of them decodes) and u in [0, 5000],
    random block tables; both launch paths against the oracle, stopping at the
    first failure (the draw is printed before it runs)."""
    import torch
    from oracle import oracle
    from paper_2606_05933_amd import workload
    from paper_2606_05933_amd.device import DeviceBatch, bits_of
    rng = np.random.default_rng(2606)
    for k in range(100):
        G = int(rng.integers(1, 17))
        hkv = int(rng.choice([1, 2, 4, 8]))
        d = int(rng.choice([64, 128]))
        n = int(rng.integers(1, 7))
        c = [1 if rng.random() < 0.33 else int(rng.integers(0, 301)) for _ in range(n)]
        u = [int(rng.integers(0, 5001)) for _ in range(n)]
        if sum(c) == 0:
            c[0] = 1
        b = workload.make_batch(workload.Shape(G * hkv, hkv, d), c, u, seed=k, spare_pages=5,
                                name=f"draw{k}")
        say(f"[gpu draw {k}] G={G} hkv={hkv} d={d} c={c} u={u}")
        kc, vc = oracle.batch_kv_append(b)
        ref, _ = oracle.batch_attention(b, kc, vc)
        db = DeviceBatch(b)
        db.step()
        torch.cuda.synchronize()
        assert np.array_equal(bits_of(db.k_cache).reshape(kc.shape), kc), f"draw {k}: K pool"
        assert np.array_equal(bits_of(db.v_cache).reshape(vc.shape), vc), f"draw {k}: V pool"
        assert_close(db.out_f32(), ref, f"draw {k}")
        two = db.out.clone()
        fz = DeviceBatch(b)
        fz.step_fused()
        torch.cuda.synchronize()
        assert np.array_equal(bits_of(fz.k_cache).reshape(kc.shape), kc), f"draw {k}: fused K pool"
        assert torch.equal(fz.out.view(torch.int16), two.view(torch.int16)), f"draw {k}: fused"
        assert db.status() == 0 and fz.status() == 0


def test_request_order_permutation_permutes_the_rows(torch_dev):
    """Reordering the requests of a batch (their rows, block-table rows and
    lengths) reorders the output rows and changes no byte of them: each
    request's work items and merge order depend only on its own (c, u)."""
    import torch
    from paper_2606_05933_amd import workload
    from paper_2606_05933_amd.device import DeviceBatch
    b = workload.make_workload("multi", seed=5)
    perm = np.random.default_rng(77).permutation(b.num_reqs)
    pb = workload.sub_batch(b, perm)
    outs = []
    for x in (b, pb):
        db = DeviceBatch(x)
        db.step_fused()
        torch.cuda.synchronize()
        assert db.status() == 0
        outs.append(db.out.view(torch.int16).cpu().numpy())
        del db
    starts = np.concatenate([[0], np.cumsum(b.q_len)])
    rows = np.concatenate([np.arange(starts[i], starts[i + 1]) for i in perm])
    assert np.array_equal(outs[1], outs[0][rows])


def test_timed_launches_stamp_the_kernels_and_match_untimed(torch_dev):
    """The timed entry points do the same work (bitwise) and stamp both events
    with a positive kernel duration."""
    import torch
    from paper_2606_05933_amd import workload
    b = workload.make_workload("l8b", seed=3)
    db = run(b)
    ref = db.out.clone()
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    for e in evs:
        e.record()  # creates the HIP events
    torch.cuda.synchronize()
    db.out.zero_()
    db.kv_append(events=(evs[0], evs[1]))
    db.attention(events=(evs[2], evs[3]))
    torch.cuda.synchronize()
    assert torch.equal(db.out.view(torch.int16), ref.view(torch.int16))
    t_app, t_att = evs[0].elapsed_time(evs[1]), evs[2].elapsed_time(evs[3])
    say(f"    kv_append {t_app * 1e3:.1f} us, attention {t_att * 1e3:.1f} us")
    assert 0 < t_app < 1000 and 0 < t_att < 1000
    assert evs[1].elapsed_time(evs[2]) >= 0


def fused_parity(b, tuning=None, plan_on_device=False):
    """ssa_append_attention on a fresh batch (new slots NaN-poisoned): the pool
    image bit for bit, outputs against the oracle, and bitwise the same as the
    two launches."""
    import torch
    from oracle import oracle
    from paper_2606_05933_amd.device import DeviceBatch, bits_of
    say(f"[gpu fused] {b.name} reqs={b.num_reqs} T={b.num_tokens} hq/hkv/d={b.shape.hq}/"
        f"{b.shape.hkv}/{b.shape.d} seed={b.seed}")
    db = DeviceBatch(b, tuning, plan_on_device=plan_on_device)
    db.step_fused()
    torch.cuda.synchronize()
    kc, vc = oracle.batch_kv_append(b)
    assert np.array_equal(bits_of(db.k_cache).reshape(kc.shape), kc), "K pool image differs"
    assert np.array_equal(bits_of(db.v_cache).reshape(vc.shape), vc), "V pool image differs"
    ref, _ = oracle.batch_attention(b, kc, vc)
    assert_close(db.out_f32(), ref, b.name + " fused")
    assert db.status() == 0, f"status word {db.status()}"
    assert not db.launch_words().any()
    fused = db.out.clone()
    two = DeviceBatch(b, tuning, plan_on_device=plan_on_device)
    two.step()
    torch.cuda.synchronize()
    assert torch.equal(fused.view(torch.int16), two.out.view(torch.int16)), "fused != two launches"
    return db


@pytest.mark.parametrize("case", range(len(SMALL)))
def test_fused_small_batches(torch_dev, case):
    hq, hkv, d, cu = SMALL[case]
    fused_parity(small(hq, hkv, d, cu, seed=case, name=f"small{case}"))


@pytest.mark.parametrize("name", ["tiny", "l8b", "multi"])
def test_fused_workloads(torch_dev, name):
    from paper_2606_05933_amd import workload
    fused_parity(workload.make_workload(name, seed=1))


def test_fused_with_splits_and_device_plan(torch_dev):
    from paper_2606_05933_amd import ssa
    b = small(32, 8, 128, [(300, 1500), (1, 3000), (1, 5000), (64, 0)], seed=5, name="fused-split")
    fused_parity(b, ssa.make_tuning(chunk_split_keys=512, decode_split_keys=1024),
                 plan_on_device=True)


def test_fused_repeated_from_poisoned_pools(torch_dev):
    """Every launch starts from the pools with the new slots NaN-poisoned, so a
    read of a new row before its append shows; the counters end at zero."""
    import torch
    from paper_2606_05933_amd import ssa, workload
    from paper_2606_05933_amd.device import DeviceBatch
    b = workload.make_workload("multi", seed=6)
    db = DeviceBatch(b, ssa.make_tuning(decode_split_keys=1024))
    k0, v0 = db.k_cache.clone(), db.v_cache.clone()
    db.step()
    torch.cuda.synchronize()
    ref = db.out.clone()
    for k in range(20):
        db.k_cache.copy_(k0)
        db.v_cache.copy_(v0)
        db.out.zero_()
        db.replan_host()
        db.step_fused()
        torch.cuda.synchronize()
        assert torch.equal(db.out.view(torch.int16), ref.view(torch.int16)), k
    assert not db.launch_words().any()


def test_fused_wait_time_out_is_reported_and_every_workgroup_exits(torch_dev):
    """The fused launch's wait for appended rows is bounded.  Forced from the
    host (the appended-rows counter preset far below zero, so the count never
    arrives within the launch, and a wait of 64 polls), every chunk item gives
    up, the launch still completes, the status word says so, and the counters
    end where they started (the last chunk item subtracts the launch's counts).
    No kernel faults or hangs: every wait has an exit."""
    import torch
    from paper_2606_05933_amd import ssa, workload
    from paper_2606_05933_amd.device import DeviceBatch
    b = workload.make_workload("tiny", seed=2)
    db = DeviceBatch(b, ssa.make_tuning(append_wait_polls=64))
    assert db.info.num_chunk_items > 0 and db.info.num_append_segments > 0
    preset = -(1 << 20)
    db.workspace[0:4].view(torch.int32).fill_(preset)
    torch.cuda.synchronize()
    db.step_fused()
    st = db.status()
    say(f"    status after the forced time-out: {st}")
    assert st & ssa.SSA_STATUS_WAIT_TIMEOUT
    words = db.launch_words()
    assert words[0] == preset and words[1] == 0
    # cleared, the same workspace serves a normal launch again
    db.workspace.zero_()
    db.plan(ssa.make_tuning())
    db.step_fused()
    assert db.status() == 0 and not db.launch_words().any()
