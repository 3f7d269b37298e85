"""Pins of the layer oracle (``oracle/layer.py``) against closed forms, and of the
library's rotary table against the oracle's angles.  No GPU.

RoPE: position 0 is the identity; every (i, i + D/2) pair keeps its norm;
rotations compose (rope(rope(x, a), b) = rope(x, a + b)); q . k of rotated heads
depends on the positions only through their difference; a D = 4 case by hand.
RMSNorm and SwiGLU: closed forms.  The linear layer: sums written out by loops.
"""
import numpy as np
import pytest

from oracle import layer as orc
from paper_2606_05933_amd import ssa


def test_positions_by_hand():
    assert list(orc.positions([3, 1, 0, 2], [5, 9, 4, 0])) == [5, 6, 7, 9, 0, 1]


def test_rope_position_zero_is_the_identity():
    x = np.random.default_rng(0).normal(size=(3, 4, 128))
    assert np.array_equal(orc.rope(x, [0, 0, 0]), x)


def test_rope_keeps_pair_norms_and_composes():
    rng = np.random.default_rng(1)
    x = rng.normal(size=(5, 2, 64))
    a, b = rng.integers(0, 40000, size=5), rng.integers(0, 40000, size=5)
    y = orc.rope(x, a)
    pair = lambda z: z[..., :32] ** 2 + z[..., 32:] ** 2
    assert np.allclose(pair(y), pair(x), rtol=1e-12)
    assert np.allclose(orc.rope(y, b), orc.rope(x, a + b), atol=1e-9)


def test_rope_scores_depend_on_the_position_difference():
    rng = np.random.default_rng(2)
    q, k = rng.normal(size=(1, 1, 128)), rng.normal(size=(1, 1, 128))
    for m, n in ((10, 3), (5000, 4993), (123, 116)):
        s = np.sum(orc.rope(q, [m]) * orc.rope(k, [n]))
        assert s == pytest.approx(np.sum(orc.rope(q, [m - n]) * k), rel=1e-9)


def test_rope_worked_by_hand():
    # D = 4: pairs (0, 2) at angle p and (1, 3) at angle p * base^(-1/2)
    base, p = 10000.0, 3
    x = np.array([[[1.0, 2.0, 3.0, 4.0]]])
    a0, a1 = p * 1.0, p * base ** -0.5
    want = [1 * np.cos(a0) - 3 * np.sin(a0), 2 * np.cos(a1) - 4 * np.sin(a1),
            3 * np.cos(a0) + 1 * np.sin(a0), 4 * np.cos(a1) + 2 * np.sin(a1)]
    assert np.allclose(orc.rope(x, [p], base)[0, 0], want, rtol=1e-15)


def test_library_rope_table_matches_the_oracle_angles():
    tab = ssa.rope_cos_sin(40000, 128)
    x = np.zeros((1, 1, 128))
    x[0, 0, :64] = 1.0  # (1, 0) pairs: the rotation's (cos, sin)
    for p in (0, 1, 777, 39999):
        r = orc.rope(x, [p])[0, 0]
        assert np.allclose(tab[p, :64], r[:64], atol=6e-8, rtol=0)
        assert np.allclose(tab[p, 64:], r[64:], atol=6e-8, rtol=0)


def test_library_rope_table_rejects_bad_arguments():
    import ctypes
    out = np.zeros((4, 8), dtype=np.float32)
    f = ssa.LIB.ssa_rope_table
    assert f(4, 8, 10000.0, None) == ssa.SSA_ERR_NULL
    for mp, d, base in ((0, 8, 1e4), (4, 7, 1e4), (4, 0, 1e4), (4, 8, 1.0), (4, 8, float("inf")),
                        (4, 8, float("nan"))):
        assert f(mp, d, base, out.ctypes.data) == ssa.SSA_ERR_ARG, (mp, d, base)
    assert not out.any()  # nothing written on an error
    assert f(4, 8, 10000.0, out.ctypes.data) == ssa.SSA_OK
    assert out[0, :4].tolist() == [1.0] * 4 and out[0, 4:].tolist() == [0.0] * 4


def test_rms_norm_and_silu_closed_forms():
    w = np.linspace(0.5, 2.0, 8)
    assert np.allclose(orc.rms_norm(np.full(8, 3.0), w, eps=0.0), w, rtol=1e-15)
    assert np.allclose(orc.rms_norm(np.full(8, -2.0), w, eps=0.0), -w, rtol=1e-15)
    assert orc.silu_mul(0.0, 5.0) == 0.0
    assert orc.silu_mul(1.0, 2.0) == pytest.approx(2.0 / (1.0 + np.exp(-1.0)), rel=1e-15)
    assert orc.silu_mul(-50.0, 1.0) == pytest.approx(-50.0 * np.exp(-50.0), rel=1e-9)


def test_linear_by_loops():
    rng = np.random.default_rng(3)
    x, w = rng.normal(size=(3, 5)), rng.normal(size=(4, 5))
    want = np.array([[sum(x[i, k] * w[j, k] for k in range(5)) for j in range(4)]
                     for i in range(3)])
    assert np.allclose(orc.linear(x, w), want, rtol=1e-13, atol=1e-13)
    assert orc.linear(x, w).shape == (3, 4)  # not the transposed product


def test_library_gate_up_interleave_is_a_row_permutation():
    i, k = 64, 3
    g = np.arange(i * k).reshape(i, k)
    u = -np.arange(i * k).reshape(i, k) - 1
    wgu = ssa.interleave_gate_up(g, u)
    for b in range(i // 16):
        assert np.array_equal(wgu[32 * b:32 * b + 16], g[16 * b:16 * b + 16])
        assert np.array_equal(wgu[32 * b + 16:32 * b + 32], u[16 * b:16 * b + 16])


# ---- the composed decoder layer (oracle.layer.decoder_layer)

def test_bf16_round_ties_and_a_bit_level_rounding():
    assert orc.bf16_round(1.0) == 1.0
    assert orc.bf16_round(1 + 2.0 ** -8) == 1.0                   # tie -> even mantissa
    assert orc.bf16_round(1 + 3 * 2.0 ** -8) == 1 + 2.0 ** -6      # tie -> even mantissa
    assert orc.bf16_round(1 + 0.6 * 2.0 ** -7) == 1 + 2.0 ** -7
    assert orc.bf16_round(-(1 + 3 * 2.0 ** -8)) == -(1 + 2.0 ** -6)
    # float32 inputs are exact in float64, so one rounding: the integer trick on
    # the float32 bits must agree everywhere
    from dense_ref import to_bf16, to_f32
    x = np.random.default_rng(4).standard_normal(200000).astype(np.float32) * 37.0
    want = to_f32(to_bf16(x)).astype(np.float64)
    assert np.array_equal(orc.bf16_round(x.astype(np.float64)), want)
    assert np.array_equal(orc.bf16_bits(want), to_bf16(want.astype(np.float32)))


SMALL = dict(hidden=256, inter=256, hq=4, hkv=2, d=64)


def small_layer(seed, q_len, ctx_len, zero=()):
    from paper_2606_05933_amd import workload
    s = SMALL
    w = workload.layer_weights(seed, s["hidden"], s["inter"], s["hq"], s["hkv"], s["d"])
    for name in zero:
        w[name] = np.zeros_like(w[name])
    b = workload.make_batch(workload.Shape(s["hq"], s["hkv"], s["d"]), q_len, ctx_len,
                            seed=seed, spare_pages=3)
    x = workload.normal_bf16((b.num_tokens, s["hidden"]), seed + 99)
    return w, b, x


def run_layer(w, b, x, q_len=None, ctx_len=None, k_cache=None, v_cache=None):
    s = SMALL
    return orc.decoder_layer(x, w, s["hq"], s["hkv"], s["d"],
                             b.q_len if q_len is None else q_len,
                             b.ctx_len if ctx_len is None else ctx_len, b.block_table,
                             b.k_cache if k_cache is None else k_cache,
                             b.v_cache if v_cache is None else v_cache, eps=1e-5)


def test_layer_with_zero_output_projections_is_the_identity():
    w, b, x = small_layer(1, [5, 1, 1], [0, 7, 40], zero=("w_o", "w_down"))
    out, _, _ = run_layer(w, b, x)
    assert np.array_equal(out, orc.from_bits(x))


def test_layer_is_causal_and_requests_are_independent():
    w, b, x = small_layer(2, [6, 1, 4], [3, 20, 0])
    out, _, _ = run_layer(w, b, x)
    x2 = x.copy()
    x2[5] ^= np.uint16(0x0040)  # the last token of request 0
    out2, _, _ = run_layer(w, b, x2)
    assert np.array_equal(out2[:5], out[:5]) and np.array_equal(out2[6:], out[6:])
    assert not np.array_equal(out2[5], out[5])
    x3 = x.copy()
    x3[7:] = x3[7:][::-1]  # request 2's rows
    out3, _, _ = run_layer(w, b, x3)
    assert np.array_equal(out3[:7], out[:7])


def test_layer_chunked_prefill_equals_one_pass():
    w, b, x = small_layer(3, [24], [10])
    out, kc, vc = run_layer(w, b, x)
    o1, kc1, vc1 = run_layer(w, b, x[:16], q_len=[16], ctx_len=[10])
    o2, kc2, vc2 = run_layer(w, b, x[16:], q_len=[8], ctx_len=[26], k_cache=kc1, v_cache=vc1)
    assert np.array_equal(np.concatenate([o1, o2]), out)
    assert np.array_equal(kc2, kc) and np.array_equal(vc2, vc)
