"""GPU parity of ssa_rope_append and ssa_layer_forward (include/ssa_layer.h)
with the CPU oracles.

Bars:
* rotated queries and keys within bf16 rounding of the float64 rotation
  (|err| <= 2^-8 |ref| + 1e-6);
* the value pool bit for bit, and every pool byte outside the new slots
  untouched;
* RoPE + append, then ssa_mixed_attention, within the attention bar
  (max 2e-2, mean 2e-3) of the attention oracle run on the oracle's own rotated
  inputs;
* ssa_layer_forward (a Llama-style decoder layer) against the composed float64
  oracle with bf16 tensors at the same places: |err| <= 2^-5 (|ref| + 1),
  mean <= 3e-3; appended keys and values within two bf16 steps.
"""
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def torch_dev():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    torch.cuda.set_device(0)
    return torch


CASES = [
    (8, 8, 64, [(64, 192), (1, 128), (1, 256), (1, 384), (1, 512)]),       # the tiny mix
    (32, 8, 128, [(17, 0), (1, 0), (33, 31), (0, 0), (1, 47), (300, 700)]),
    (28, 4, 128, [(100, 1000), (1, 4095), (1, 16), (513, 7)]),
    (64, 8, 128, [(40, 30000), (1, 32767)]),                                # long positions
]


def run_case(torch, hq, hkv, d, cu, seed):
    from dense_ref import to_bf16, to_f32
    from oracle import layer as olay
    from oracle import oracle as orc
    from paper_2606_05933_amd import ssa, workload
    from paper_2606_05933_amd.device import DeviceBatch, bits_of
    shape = workload.Shape(hq, hkv, d)
    b = workload.make_batch(shape, [c for c, _ in cu], [u for _, u in cu], seed=seed,
                            spare_pages=7, name="rope")
    say(f"[gpu rope] hq/hkv/d={hq}/{hkv}/{d} reqs={b.num_reqs} T={b.num_tokens} seed={seed}")
    T = b.num_tokens
    qkv = np.concatenate([b.q, b.k_new, b.v_new], axis=1).reshape(T, -1)
    max_pos = int(max(u + c for c, u in cu)) + 3
    db = DeviceBatch(b)
    qkv_t = torch.from_numpy(qkv.view(np.int16)).cuda().view(torch.bfloat16)
    cos_t = torch.from_numpy(ssa.rope_cos_sin(max_pos, d)).cuda()
    q_out = torch.zeros((T, hq, d), dtype=torch.bfloat16, device="cuda")
    ssa.rope_append(db.shape, db.plan_host, db.plan_dev, qkv_t, cos_t, q_out, db.k_cache,
                    db.v_cache, db.block_table)
    torch.cuda.synchronize()
    pos = olay.positions(b.q_len, b.ctx_len)
    q_ref = olay.rope(to_f32(b.q).astype(np.float64), pos)
    k_ref = olay.rope(to_f32(b.k_new).astype(np.float64), pos)
    q_got = to_f32(bits_of(q_out).reshape(T, hq, d)).astype(np.float64)
    assert np.all(np.abs(q_got - q_ref) <= 2.0 ** -8 * np.abs(q_ref) + 1e-6)
    # pools: the values bit for bit and every byte outside the new slots untouched
    kc = bits_of(db.k_cache).reshape(b.k_cache.shape)
    vc = bits_of(db.v_cache).reshape(b.v_cache.shape)
    _, vc_ref = orc.kv_append(hkv, d, 16, b.q_len, b.ctx_len, b.block_table, b.k_new, b.v_new,
                              b.k_cache, b.v_cache)
    assert np.array_equal(vc, vc_ref)
    new = np.zeros(b.k_cache.shape, dtype=bool)
    t = 0
    for i, (c, u) in enumerate(zip(b.q_len, b.ctx_len)):
        for j in range(int(c)):
            p = int(u) + j
            page, slot = int(b.block_table[i, p // 16]), p % 16
            new[page, :, slot, :] = True
            got = to_f32(kc[page, :, slot, :]).astype(np.float64)
            ref = k_ref[t]
            assert np.all(np.abs(got - ref) <= 2.0 ** -8 * np.abs(ref) + 1e-6), (i, j)
            t += 1
    assert np.array_equal(kc[~new], b.k_cache[~new])
    return b, db, q_out, q_ref, k_ref


@pytest.mark.parametrize("case", range(len(CASES)))
def test_rope_append_matches_the_oracle(torch_dev, case):
    hq, hkv, d, cu = CASES[case]
    run_case(torch_dev, hq, hkv, d, cu, seed=case)


@pytest.mark.parametrize("case", range(len(CASES)))
def test_rope_append_then_attention(torch_dev, case):
    from dense_ref import to_bf16
    from oracle import oracle as orc
    torch = torch_dev
    hq, hkv, d, cu = CASES[case]
    b, db, q_out, q_ref, k_ref = run_case(torch, hq, hkv, d, cu, seed=10 + case)
    db.q.copy_(q_out)
    db.attention()
    torch.cuda.synchronize()
    kc_ref, vc_ref = orc.kv_append(hkv, d, 16, b.q_len, b.ctx_len, b.block_table,
                                   to_bf16(k_ref.astype(np.float32)), b.v_new, b.k_cache,
                                   b.v_cache)
    ref, _ = orc.attention(hq, hkv, d, 16, b.shape.softmax_scale, b.q_len, b.ctx_len,
                           b.block_table, to_bf16(q_ref.astype(np.float32)), kc_ref, vc_ref)
    got = db.out_f32().astype(np.float64)
    err = np.abs(got - ref)
    say(f"    rope+attention: max_abs={err.max():.3e} mean_abs={err.mean():.3e}")
    assert np.isfinite(got).all()
    assert err.max() <= 2e-2 and err.mean() <= 2e-3


def test_rope_append_rejects_positions_past_the_table(torch_dev):
    from paper_2606_05933_amd import ssa, workload
    from paper_2606_05933_amd.device import DeviceBatch
    torch = torch_dev
    b = workload.make_batch(workload.Shape(8, 8, 64), [4, 1], [10, 20], seed=0, spare_pages=2)
    db = DeviceBatch(b)
    qkv = torch.zeros((b.num_tokens, 24 * 64), dtype=torch.bfloat16, device="cuda")
    q_out = torch.zeros((b.num_tokens, 8, 64), dtype=torch.bfloat16, device="cuda")
    short = torch.from_numpy(ssa.rope_cos_sin(20, 64)).cuda()  # position 20 needs 21 rows
    before = db.k_cache.clone()
    with pytest.raises(ssa.SsaError):
        ssa.rope_append(db.shape, db.plan_host, db.plan_dev, qkv, short, q_out, db.k_cache,
                        db.v_cache, db.block_table)
    torch.cuda.synchronize()
    assert torch.equal(before.view(torch.int16), db.k_cache.view(torch.int16))  # NaN-poisoned


# ---- ssa_layer_forward: one decoder layer against the composed oracle

LAYER_CASES = [
    # hidden, inter, hq, hkv, d, [(c, u), ...], out written over x
    (256, 256, 4, 2, 64, [(20, 30), (1, 100), (1, 5), (37, 0)], False),
    (4096, 14336, 32, 8, 128, [(64, 192), (1, 1000), (1, 4000), (1, 17), (70, 0)], False),
    (4096, 14336, 32, 8, 128, [(1, u) for u in (3, 90, 700, 2500, 6000)], True),  # decodes only
    (512, 1024, 8, 8, 64, [(150, 0), (33, 260)], True),                            # prefill only
]


@pytest.mark.parametrize("case", range(len(LAYER_CASES)))
def test_layer_forward_matches_the_oracle(torch_dev, case):
    from dense_ref import to_f32
    from oracle import layer as olay
    from paper_2606_05933_amd import ssa, workload
    from paper_2606_05933_amd.device import DeviceBatch, bits_of
    torch = torch_dev
    hidden, inter, hq, hkv, d, cu, in_place = LAYER_CASES[case]
    seed = 40 + case
    w = workload.layer_weights(seed, hidden, inter, hq, hkv, d)
    b = workload.make_batch(workload.Shape(hq, hkv, d), [c for c, _ in cu], [u for _, u in cu],
                            seed=seed, spare_pages=5, name="layer")
    T = b.num_tokens
    say(f"[gpu layer] hidden={hidden} inter={inter} hq/hkv/d={hq}/{hkv}/{d} T={T} seed={seed} "
        f"in_place={in_place}")
    x = workload.normal_bf16((T, hidden), seed + 99)
    db = DeviceBatch(b)
    lw = ssa.LayerWeights(w, hq, hkv, d, max_position=int(max(c + u for c, u in cu)) + 1)
    ws = torch.zeros(ssa.layer_workspace_size(db.shape, db.plan_host, lw), dtype=torch.uint8,
                     device="cuda")
    xd = torch.from_numpy(x.view(np.int16)).cuda().view(torch.bfloat16)
    out = xd if in_place else torch.full((T, hidden), float("nan"), dtype=torch.bfloat16,
                                         device="cuda")
    ssa.layer_forward(db.shape, db.plan_host, db.plan_dev, lw, xd, out, db.k_cache, db.v_cache,
                      db.block_table, ws)
    torch.cuda.synchronize()
    ref, kc_ref, vc_ref = olay.decoder_layer(x, w, hq, hkv, d, b.q_len, b.ctx_len,
                                             b.block_table, b.k_cache, b.v_cache, eps=1e-5)
    got = to_f32(bits_of(out).reshape(T, hidden)).astype(np.float64)
    err = np.abs(got - ref)
    rel = err / (np.abs(ref) + 1.0)
    say(f"    out: max_abs={err.max():.3e} mean_abs={err.mean():.3e} max_rel1={rel.max():.3e} "
        f"rms_ref={np.sqrt(np.mean(ref ** 2)):.3f}")
    # the new pool slots: within a few bf16 rounding steps of the oracle's
    kc = to_f32(bits_of(db.k_cache).reshape(b.k_cache.shape)).astype(np.float64)
    vc = to_f32(bits_of(db.v_cache).reshape(b.v_cache.shape)).astype(np.float64)
    kr, vr = to_f32(kc_ref).astype(np.float64), to_f32(vc_ref).astype(np.float64)
    fin = np.isfinite(kr)
    vfin = np.isfinite(vr)
    kerr, verr = np.abs(kc[fin] - kr[fin]), np.abs(vc[vfin] - vr[vfin])
    say(f"    pools: k max_abs={kerr.max():.3e} v max_abs={verr.max():.3e}")
    assert np.array_equal(np.isfinite(kc), fin)  # no slot outside the new ones written
    assert np.isfinite(got).all()
    # Seven bf16 tensors lie between x and out; each may round one step apart
    # from the oracle's (fp32 vs fp64 sums), and the residual stream carries
    # such steps with gain about one: a few bf16 steps at unit scale.
    assert np.all(err <= 2.0 ** -5 * (np.abs(ref) + 1.0)) and err.mean() <= 3e-3
    # the appended keys and values: at most two rounding steps apart; a key
    # pair (i, i + D/2) is rotated together, which spreads a rounding step of
    # one member over both and keeps the pair's norm
    half = d // 2
    pn = np.sqrt(kr[..., :half] ** 2 + kr[..., half:] ** 2)
    pn = np.concatenate([pn, pn], axis=-1)
    assert np.all(kerr <= 2.0 ** -6 * pn[fin] + 2.0 ** -10)
    assert np.all(verr <= 2.0 ** -6 * np.abs(vr[vfin]) + 2.0 ** -10)


def test_layer_forward_replays_from_a_hip_graph(torch_dev):
    """ssa_layer_forward captured in a HIP graph (eight launches, no allocation,
    no memset) replays to the eager result, bit for bit, with eager work and
    synchronisations between the replays."""
    from paper_2606_05933_amd import ssa, workload
    from paper_2606_05933_amd.device import DeviceBatch
    torch = torch_dev
    hidden, inter, hq, hkv, d = 512, 1024, 8, 2, 64
    cu = [(40, 100), (1, 300), (1, 7), (17, 0)]
    w = workload.layer_weights(60, hidden, inter, hq, hkv, d)
    b = workload.make_batch(workload.Shape(hq, hkv, d), [c for c, _ in cu], [u for _, u in cu],
                            seed=60, spare_pages=5, name="graph")
    T = b.num_tokens
    say(f"[gpu layer graph] T={T}")
    db = DeviceBatch(b)
    lw = ssa.LayerWeights(w, hq, hkv, d, max_position=400)
    ws = torch.zeros(ssa.layer_workspace_size(db.shape, db.plan_host, lw), dtype=torch.uint8,
                     device="cuda")
    x = torch.from_numpy(workload.normal_bf16((T, hidden), 61).view(np.int16)).cuda().view(
        torch.bfloat16)
    out = torch.empty_like(x)
    kc0, vc0 = db.k_cache.clone(), db.v_cache.clone()

    def layer():
        ssa.layer_forward(db.shape, db.plan_host, db.plan_dev, lw, x, out, db.k_cache,
                          db.v_cache, db.block_table, ws)

    layer()
    torch.cuda.synchronize()
    eager = out.clone()
    kc1, vc1 = db.k_cache.clone(), db.v_cache.clone()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        layer()  # warm the stream before capture
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        layer()
    for k in range(4):
        out.zero_()
        db.k_cache.copy_(kc0)
        db.v_cache.copy_(vc0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), eager.view(torch.int16)), k
        assert torch.equal(db.k_cache.view(torch.int16), kc1.view(torch.int16)), k
        assert torch.equal(db.v_cache.view(torch.int16), vc1.view(torch.int16)), k
        layer()  # eager work between replays
        torch.cuda.synchronize()
