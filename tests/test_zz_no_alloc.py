"""The allocation-free fused launch (ssa_append_attention_static) against the
workspace one (ssa_append_attention), through the C ABI, on an MI355X: two
calls in a row, the second on a smaller batch, each on fresh (poisoned)
pools.  Pool images and outputs must be identical bit for bit (the same
kernels), and the outputs within the oracle's bars."""
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def static_vs_workspace(b):
    import torch
    from oracle import oracle
    from paper_2606_05933_amd import ssa
    from paper_2606_05933_amd.device import DeviceBatch, bits_of
    say(f"[gpu static] {b.name} reqs={b.num_reqs} T={b.num_tokens} "
        f"hq/hkv/d={b.shape.hq}/{b.shape.hkv}/{b.shape.d} seed={b.seed}")
    ref = DeviceBatch(b)
    ref.step_fused()
    torch.cuda.synchronize()
    assert ref.status() == 0
    db = DeviceBatch(b)
    ssa.append_attention_static(db.shape, db.plan_host, db.plan_dev, db.q, db.k_new, db.v_new,
                                db.k_cache, db.v_cache, db.block_table, db.out)
    torch.cuda.synchronize()
    assert torch.equal(db.out.view(torch.int16), ref.out.view(torch.int16)), "outputs differ"
    assert torch.equal(db.k_cache.view(torch.int16), ref.k_cache.view(torch.int16))
    assert torch.equal(db.v_cache.view(torch.int16), ref.v_cache.view(torch.int16))
    kc, vc = oracle.batch_kv_append(b)
    assert np.array_equal(bits_of(db.k_cache).reshape(kc.shape), kc), "K pool image differs"
    out, _ = oracle.batch_attention(b, kc, vc)
    err = np.abs(db.out_f32().astype(np.float64) - out)
    say(f"    max_abs={err.max():.3e} mean_abs={err.mean():.3e}")
    assert np.isfinite(db.out_f32()).all()
    assert err.max() <= 2e-2 and err.mean() <= 2e-3


def test_static_scratch_matches_workspace_launch_twice_then_smaller():
    import torch
    from paper_2606_05933_amd import ssa, workload
    assert torch.cuda.is_available()
    torch.cuda.set_device(0)
    # first a batch with merge groups (chunk and decode splits), then a smaller one
    big = workload.make_batch(workload.Shape(32, 8, 128),
                              [300, 1, 1, 64, 1], [1500, 3000, 5000, 0, 9000], seed=5,
                              name="static-big")
    static_vs_workspace(big)
    small = workload.make_workload("tiny", seed=3)
    static_vs_workspace(small)
    # a plan larger than the scratch is refused before any launch
    huge_q, huge_u = [1] * 4, [1 << 20] * 4
    shape = ssa.make_shape(64, 8, 128, 1 << 20, (1 << 20) // 16 + 1, 0.0884)
    pb, wb = ssa.ssa_plan_size(shape, huge_q, huge_u)
    assert wb > (32 << 20)
    blob, _ = ssa.ssa_plan(shape, huge_q, huge_u)
    rc = ssa.LIB.ssa_append_attention_static(
        ssa.ctypes.byref(shape), blob.ctypes.data, blob.ctypes.data, *([None] * 10))
    assert rc == -8
