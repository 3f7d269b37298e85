"""The allocation-free fused launch (ssa_append_attention_static) captured in a
HIP graph, the use it exists for: the graph is replayed several times, with
eager work and synchronisations between the replays, and every replay must
give the eager launch's outputs and pool images bit for bit.  The scratch's
one-time set-up (its device address) happens in an eager call before the
capture."""
import sys

import pytest

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def test_static_launch_replays_from_a_graph():
    import torch
    from paper_2606_05933_amd import ssa, workload
    from paper_2606_05933_amd.device import DeviceBatch
    assert torch.cuda.is_available()
    torch.cuda.set_device(0)
    # chunk and decode splits, so the launch uses merge tickets in the scratch
    b = workload.make_batch(workload.Shape(32, 8, 128), [300, 1, 1, 64, 1],
                            [1500, 3000, 5000, 0, 9000], seed=11, name="graph")
    say(f"[gpu graph] {b.name} reqs={b.num_reqs} T={b.num_tokens}")
    ref = DeviceBatch(b)
    ref.step_fused()
    torch.cuda.synchronize()
    assert ref.status() == 0

    db = DeviceBatch(b)
    args = (db.shape, db.plan_host, db.plan_dev, db.q, db.k_new, db.v_new, db.k_cache,
            db.v_cache, db.block_table, db.out)
    ssa.append_attention_static(*args)  # eager: sets up the scratch, same bits as ref
    torch.cuda.synchronize()
    assert torch.equal(db.out.view(torch.int16), ref.out.view(torch.int16))

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            ssa.append_attention_static(*args)
    torch.cuda.synchronize()

    junk = torch.empty(1 << 20, dtype=torch.float32, device="cuda")
    for r in range(5):
        db.out.fill_(0)          # eager work between replays
        junk.uniform_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        say(f"    replay {r}")
        assert torch.equal(db.out.view(torch.int16), ref.out.view(torch.int16)), f"replay {r}"
        assert torch.equal(db.k_cache.view(torch.int16), ref.k_cache.view(torch.int16))
        assert torch.equal(db.v_cache.view(torch.int16), ref.v_cache.view(torch.int16))
    # an eager call after the replays still matches (the scratch is back at rest)
    db.out.fill_(0)
    ssa.append_attention_static(*args)
    torch.cuda.synchronize()
    assert torch.equal(db.out.view(torch.int16), ref.out.view(torch.int16))
