"""Pins of the CPU oracle against what the mathematics fixes (no GPU).

The oracle is the plain definition of mixed chunked-prefill + decode attention
over a paged cache (batch B = {(c_i, u_i)}, Sec. 3.2; chunked prefill, Sec. 1 and
Sec. 2.1).  It is pinned here by things other than itself:

* brute-force dense fp64 softmax attention over unpaged sequences (numpy);
* torch's scaled_dot_product_attention in float64 on the CPU with an explicit
  boolean mask (a library routine);
* closed forms: one visible key, zero logits, constant values, a dominant key;
* the invariants: chunking a prefill in any way, decode = last row of full
  causal attention, block-table permutation, request-order permutation,
  key shift, value affine map, GQA = MHA with repeated kv heads, independence
  of other requests;
* the kv_append image against an independent scatter, and its round trip.
"""
import numpy as np
import pytest

from dense_ref import NAN16, dense_attention, gather, page_out, to_bf16, to_f32
from oracle import oracle as orc


def draw_case(hq, hkv, d, P, cu, seed, grid=None):
    """Logical per-request sequences for the (c, u) list.  With ``grid`` the
    values are drawn from a small exact grid (multiples of 1/grid in [-2, 2])."""
    rng = np.random.default_rng(seed)

    def vals(shape):
        if grid:
            return to_bf16(rng.integers(-2 * grid, 2 * grid + 1, size=shape) / grid)
        return to_bf16(rng.standard_normal(shape).astype(np.float32))

    ks, vs, qs = [], [], []
    for c, u in cu:
        ks.append(vals((u + c, hkv, d)))
        vs.append(vals((u + c, hkv, d)))
        qs.append(vals((c, hq, d)))
    return ks, vs, qs, rng


def run_oracle(hq, hkv, d, P, scale, cu, ks, vs, qs, rng, spare=5, lib=None):
    bt, kc, vc = page_out(ks, vs, hkv, d, P, rng, spare=spare)
    q = np.concatenate(qs, axis=0) if qs else np.zeros((0, hq, d), np.uint16)
    q_len = np.array([c for c, _ in cu], np.int32)
    ctx = np.array([u for _, u in cu], np.int32)
    out, _ = orc.attention(hq, hkv, d, P, scale, q_len, ctx, bt, q, kc, vc, lib=lib)
    return out


def dense_all(hq, hkv, d, scale, cu, ks, vs, qs):
    rows = []
    for (c, u), k, v, q in zip(cu, ks, vs, qs):
        if c == 0:
            continue
        rows.append(dense_attention(to_f32(q).astype(np.float64), to_f32(k).astype(np.float64),
                                    to_f32(v).astype(np.float64), u, np.float64(np.float32(scale))))
    return np.concatenate(rows, axis=0) if rows else np.zeros((0, hq, d))


CASES = [
    # hq, hkv, d, P, [(c, u), ...]
    (2, 2, 8, 4, [(5, 0), (1, 3), (3, 6)]),
    (4, 1, 16, 16, [(1, 0), (7, 9), (1, 31), (17, 16)]),
    (8, 2, 16, 4, [(0, 5), (2, 0), (1, 1), (6, 13)]),
    (7, 1, 32, 16, [(20, 40), (1, 100)]),
    (8, 8, 64, 16, [(16, 48), (1, 128), (1, 15)]),
]


@pytest.mark.parametrize("case", CASES)
def test_oracle_matches_dense_bruteforce(case):
    hq, hkv, d, P, cu = case
    scale = float(np.float32(1.0 / np.sqrt(d)))
    ks, vs, qs, rng = draw_case(hq, hkv, d, P, cu, seed=hq * 31 + d)
    out = run_oracle(hq, hkv, d, P, scale, cu, ks, vs, qs, rng)
    ref = dense_all(hq, hkv, d, scale, cu, ks, vs, qs)
    assert out.shape == ref.shape
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)


def test_oracle_matches_torch_sdpa_float64():
    torch = pytest.importorskip("torch")
    hq, hkv, d, P = 8, 2, 32, 16
    cu = [(9, 23), (1, 40), (12, 0)]
    scale = float(np.float32(1.0 / np.sqrt(d)))
    ks, vs, qs, rng = draw_case(hq, hkv, d, P, cu, seed=5)
    out = run_oracle(hq, hkv, d, P, scale, cu, ks, vs, qs, rng)
    rows = []
    for (c, u), k, v, q in zip(cu, ks, vs, qs):
        qt = torch.from_numpy(to_f32(q).astype(np.float64)).permute(1, 0, 2)  # [Hq, c, D]
        kt = torch.from_numpy(to_f32(k).astype(np.float64)).permute(1, 0, 2)
        vt = torch.from_numpy(to_f32(v).astype(np.float64)).permute(1, 0, 2)
        kt = kt.repeat_interleave(hq // hkv, dim=0)
        vt = vt.repeat_interleave(hq // hkv, dim=0)
        mask = torch.arange(u + c)[None, :] <= (u + torch.arange(c))[:, None]
        o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask,
                                                             scale=scale)
        rows.append(o.permute(1, 0, 2).numpy())
        if u == 0:  # with no prefix the mask is the plain causal one
            o2 = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, is_causal=True,
                                                                  scale=scale)
            np.testing.assert_allclose(o2.numpy(), o.numpy(), rtol=0, atol=1e-12)
    np.testing.assert_allclose(out, np.concatenate(rows), rtol=0, atol=1e-12)


# ---------------------------------------------------------------- closed forms

def test_single_visible_key_returns_its_value_exactly():
    hq, hkv, d, P = 4, 2, 16, 16
    cu = [(1, 0), (1, 0)]
    ks, vs, qs, rng = draw_case(hq, hkv, d, P, cu, seed=1)
    out = run_oracle(hq, hkv, d, P, 0.25, cu, ks, vs, qs, rng)
    for i in range(2):
        for h in range(hq):
            assert np.array_equal(out[i, h], to_f32(vs[i][0, h // 2]).astype(np.float64))


@pytest.mark.parametrize("how", ["scale0", "q0", "kconst"])
def test_uniform_weights_give_prefix_means(how):
    hq, hkv, d, P = 4, 2, 16, 4
    cu = [(6, 5), (1, 9)]
    ks, vs, qs, rng = draw_case(hq, hkv, d, P, cu, seed=2)
    scale = 0.0 if how == "scale0" else 0.25
    if how == "q0":
        qs = [np.zeros_like(q) for q in qs]
    if how == "kconst":
        ks = [np.broadcast_to(k[:1], k.shape).copy() for k in ks]
    out = run_oracle(hq, hkv, d, P, scale, cu, ks, vs, qs, rng)
    r = 0
    for (c, u), v in zip(cu, vs):
        vf = to_f32(v).astype(np.float64)
        for j in range(c):
            for h in range(hq):
                np.testing.assert_allclose(out[r, h], vf[: u + j + 1, h // 2].mean(axis=0),
                                           rtol=0, atol=1e-12)
            r += 1


def test_constant_values_give_that_constant():
    hq, hkv, d, P = 4, 4, 16, 16
    cu = [(5, 20), (1, 3)]
    ks, vs, qs, rng = draw_case(hq, hkv, d, P, cu, seed=3)
    const = to_bf16(np.linspace(-3, 3, d).astype(np.float32))
    vs = [np.broadcast_to(const, v.shape).copy() for v in vs]
    out = run_oracle(hq, hkv, d, P, 0.25, cu, ks, vs, qs, rng)
    np.testing.assert_allclose(out, np.broadcast_to(to_f32(const), out.shape), rtol=0, atol=1e-12)


def test_dominant_key_selects_its_value():
    hq, hkv, d, P = 2, 1, 16, 4
    cu = [(1, 10)]
    ks, vs, qs, rng = draw_case(hq, hkv, d, P, cu, seed=4)
    spike = 7
    e = np.zeros(d, np.float32)
    e[3] = 64.0
    qs[0][0, :, :] = to_bf16(e)
    ks[0][spike, 0, :] = to_bf16(e)
    out = run_oracle(hq, hkv, d, P, 1.0, cu, ks, vs, qs, rng)
    np.testing.assert_allclose(out[0, 0], to_f32(vs[0][spike, 0]), rtol=0, atol=1e-12)


# ------------------------------------------------------------------ invariants

def test_chunking_a_prefill_any_way_matches_monolithic_prefill():
    hq, hkv, d, P = 4, 2, 16, 4
    L = 37
    ks, vs, qs, rng = draw_case(hq, hkv, d, P, [(L, 0)], seed=6)
    mono = run_oracle(hq, hkv, d, P, 0.25, [(L, 0)], ks, vs, qs, rng)
    for cuts in ([1, 36], [16, 16, 5], [3, 1, 1, 20, 12], [37]):
        rows, u = [], 0
        for c in cuts:
            # the iteration at prefix u computing c tokens sees keys 0..u+c-1
            o = run_oracle(hq, hkv, d, P, 0.25, [(c, u)], [ks[0][: u + c]], [vs[0][: u + c]],
                           [qs[0][u: u + c]], np.random.default_rng(u))
            rows.append(o)
            u += c
        assert np.array_equal(np.concatenate(rows), mono)


def test_decode_equals_last_row_of_full_causal_attention():
    hq, hkv, d, P = 8, 2, 16, 16
    u = 45
    ks, vs, qs, rng = draw_case(hq, hkv, d, P, [(u + 1, 0)], seed=7)
    full = run_oracle(hq, hkv, d, P, 0.25, [(u + 1, 0)], ks, vs, qs, rng)
    dec = run_oracle(hq, hkv, d, P, 0.25, [(1, u)], ks, vs, [qs[0][u:]], np.random.default_rng(1))
    assert np.array_equal(dec[0], full[-1])


def test_block_table_permutation_leaves_output_unchanged():
    hq, hkv, d, P = 4, 2, 16, 4
    cu = [(5, 11), (1, 30), (9, 0)]
    ks, vs, qs, _ = draw_case(hq, hkv, d, P, cu, seed=8)
    outs = [run_oracle(hq, hkv, d, P, 0.25, cu, ks, vs, qs, np.random.default_rng(s), spare=s)
            for s in (0, 3, 17)]
    assert np.array_equal(outs[0], outs[1]) and np.array_equal(outs[0], outs[2])


def test_request_order_permutation_permutes_rows():
    hq, hkv, d, P = 4, 2, 16, 16
    cu = [(5, 11), (1, 30), (9, 0), (1, 2)]
    ks, vs, qs, rng = draw_case(hq, hkv, d, P, cu, seed=9)
    out = run_oracle(hq, hkv, d, P, 0.25, cu, ks, vs, qs, rng)
    order = [2, 0, 3, 1]
    out2 = run_oracle(hq, hkv, d, P, 0.25, [cu[i] for i in order], [ks[i] for i in order],
                      [vs[i] for i in order], [qs[i] for i in order], np.random.default_rng(3))
    starts = np.concatenate([[0], np.cumsum([c for c, _ in cu])])
    expect = np.concatenate([out[starts[i]: starts[i + 1]] for i in order])
    assert np.array_equal(out2, expect)


def test_other_requests_do_not_change_a_requests_rows():
    hq, hkv, d, P = 4, 4, 16, 4
    cu = [(7, 9), (1, 33), (3, 2)]
    ks, vs, qs, rng = draw_case(hq, hkv, d, P, cu, seed=10)
    out = run_oracle(hq, hkv, d, P, 0.25, cu, ks, vs, qs, rng)
    alone = run_oracle(hq, hkv, d, P, 0.25, cu[1:2], ks[1:2], vs[1:2], qs[1:2],
                       np.random.default_rng(5))
    assert np.array_equal(alone[0], out[7])


def test_key_shift_per_kv_head_leaves_output_unchanged():
    # exact grid values: k + delta stays exactly representable in bf16
    hq, hkv, d, P = 4, 2, 16, 4
    cu = [(6, 10), (1, 21)]
    ks, vs, qs, rng = draw_case(hq, hkv, d, P, cu, seed=11, grid=4)
    out = run_oracle(hq, hkv, d, P, 0.125, cu, ks, vs, qs, rng)
    delta = np.random.default_rng(1).integers(-8, 9, size=(hkv, d)) / 4.0
    ks2 = [to_bf16(to_f32(k) + delta[None].astype(np.float32)) for k in ks]
    assert all(np.array_equal(to_f32(a), to_f32(b) + delta[None].astype(np.float32))
               for a, b in zip(ks2, ks))
    out2 = run_oracle(hq, hkv, d, P, 0.125, cu, ks2, vs, qs, np.random.default_rng(2))
    np.testing.assert_allclose(out2, out, rtol=0, atol=1e-12)


def test_value_affine_map_commutes():
    hq, hkv, d, P = 4, 2, 16, 4
    cu = [(6, 10), (1, 21)]
    ks, vs, qs, rng = draw_case(hq, hkv, d, P, cu, seed=12, grid=4)
    out = run_oracle(hq, hkv, d, P, 0.25, cu, ks, vs, qs, rng)
    a, b = 2.0, 0.5
    vs2 = [to_bf16(a * to_f32(v) + b) for v in vs]
    out2 = run_oracle(hq, hkv, d, P, 0.25, cu, ks, vs2, qs, np.random.default_rng(2))
    np.testing.assert_allclose(out2, a * out + b, rtol=0, atol=1e-12)


def test_gqa_equals_mha_with_repeated_kv_heads():
    hq, hkv, d, P = 8, 2, 16, 16
    cu = [(5, 11), (1, 30)]
    ks, vs, qs, rng = draw_case(hq, hkv, d, P, cu, seed=13)
    out = run_oracle(hq, hkv, d, P, 0.25, cu, ks, vs, qs, rng)
    rep = hq // hkv
    ks2 = [np.repeat(k, rep, axis=1) for k in ks]
    vs2 = [np.repeat(v, rep, axis=1) for v in vs]
    out2 = run_oracle(hq, hq, d, P, 0.25, cu, ks2, vs2, qs, np.random.default_rng(3))
    assert np.array_equal(out, out2)


# -------------------------------------------------------------------- kv_append

def test_kv_append_image_and_round_trip():
    hq, hkv, d, P = 4, 2, 16, 4
    cu = [(5, 11), (1, 30), (9, 0), (0, 7), (1, 0)]
    ks, vs, _, rng = draw_case(hq, hkv, d, P, cu, seed=14)
    # full sequences paged out; the "before" pools poison positions >= u
    bt, kfull, vfull = page_out(ks, vs, hkv, d, P, rng, spare=3)
    kc, vc = kfull.copy(), vfull.copy()
    for i, (c, u) in enumerate(cu):
        for t in range(u, u + c):
            kc[bt[i, t // P], :, t % P, :] = NAN16
            vc[bt[i, t // P], :, :, t % P] = NAN16
    k_new = np.concatenate([k[u:] for (c, u), k in zip(cu, ks)])
    v_new = np.concatenate([v[u:] for (c, u), v in zip(cu, vs)])
    q_len = np.array([c for c, _ in cu], np.int32)
    ctx = np.array([u for _, u in cu], np.int32)
    k2, v2 = orc.kv_append(hkv, d, P, q_len, ctx, bt, k_new, v_new, kc, vc)
    assert np.array_equal(k2, kfull) and np.array_equal(v2, vfull)
    r = 0
    for i, (c, u) in enumerate(cu):
        kk, vv = gather(k2, v2, bt[i], u + c, P)
        assert np.array_equal(kk[u:], k_new[r: r + c]) and np.array_equal(vv[u:], v_new[r: r + c])
        r += c


def test_rows_entry_matches_full_entry():
    hq, hkv, d, P = 8, 2, 16, 4
    cu = [(0, 3), (6, 10), (1, 21), (0, 0), (3, 1)]
    ks, vs, qs, rng = draw_case(hq, hkv, d, P, cu, seed=15)
    bt, kc, vc = page_out(ks, vs, hkv, d, P, rng)
    q = np.concatenate(qs)
    q_len = np.array([c for c, _ in cu], np.int32)
    ctx = np.array([u for _, u in cu], np.int32)
    full, _ = orc.attention(hq, hkv, d, P, 0.25, q_len, ctx, bt, q, kc, vc)
    rows = np.repeat(np.arange(q.shape[0]), hq)
    heads = np.tile(np.arange(hq), q.shape[0])
    sel, _ = orc.attention_rows(hq, hkv, d, P, 0.25, q_len, ctx, bt, q, kc, vc, rows, heads)
    assert np.array_equal(sel.reshape(full.shape), full)
