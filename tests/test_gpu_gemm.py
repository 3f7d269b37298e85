"""GPU parity of ssa_linear and ssa_rms_norm (include/ssa_layer.h) with the
float64 oracle (oracle/layer.py) on the same bf16 inputs.

Bars (bf16 output: its rounding is at most 2^-8 |ref|):
* linear:   |got - ref| <= 2^-8 |ref| + 2^-17 S, with S = sum_k |x_k w_k| (fp32
  accumulation; a dropped or doubled 32-wide K slice is far above this);
* SwiGLU:   |got - ref| <= 2^-8 |ref| + 2^-16 (S_g |up| + S_u |silu(gate)|);
* RMSNorm:  |got - ref| <= 2^-8 |ref| + 2^-20 |x w| / rms(x).
Also: two calls in a row give the same bits (split tickets reset, partials added
in split order); the residual epilogue works in place; at full Llama-3-8B sizes
sampled rows are checked.
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


NONE, RES, SWIGLU = 0, 1, 2
CASES = [  # (M, N, K, epilogue)
    (1, 128, 64, NONE),
    (37, 256, 320, NONE),
    (130, 384, 4096, NONE),        # 6 tiles: K split 16 ways
    (300, 640, 1024, RES),
    (129, 256, 2048, SWIGLU),
    (28, 6144, 4096, NONE),        # a decode-only batch through the QKV projection
    (520, 4096, 14336, RES),       # the down projection of a mixed batch, K split 3
    (1000, 1024, 512, SWIGLU),
    (257, 28672, 4096, SWIGLU),    # gate/up projection
    # tiles that overfill the chip by part of a round
    (700, 11264, 512, RES),        # 528 tiles of 128 x 128, ragged M
    (1100, 8192, 256, NONE),       # 576 tiles, 4 K blocks each
    (640, 28672, 4096, SWIGLU),    # 1120 tiles of 128 x 128
    (1152, 28672, 4096, SWIGLU),   # 560 tiles of 256 x 256
    # where 192-row tiles fit one round of the chip and 128- or 160-row ones do not
    (370, 28672, 1024, SWIGLU),    # ragged M
    (384, 28672, 4096, NONE),
]


def dev_bf16(torch, bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(torch.bfloat16)


def inputs(m, n, k, epi, seed):
    from paper_2606_05933_amd import ssa, workload
    x = workload.normal_bf16((m, k), seed)
    if epi == SWIGLU:
        wg = workload.normal_bf16((n // 2, k), seed + 1, k ** -0.5)
        wu = workload.normal_bf16((n // 2, k), seed + 2, k ** -0.5)
        return x, (wg, wu), ssa.interleave_gate_up(wg, wu), None
    w = workload.normal_bf16((n, k), seed + 1, k ** -0.5)
    res = workload.normal_bf16((m, n), seed + 3) if epi == RES else None
    return x, w, w, res


def reference(x, w, res, epi, rows):
    """Oracle values and the error bound for the given rows."""
    from dense_ref import to_f32
    from oracle import layer as olay
    xf = to_f32(x[rows]).astype(np.float64)
    if epi == SWIGLU:
        wg, wu = (to_f32(a).astype(np.float64) for a in w)
        g, u = olay.linear(xf, wg), olay.linear(xf, wu)
        ref = olay.silu_mul(g, u)
        sg, su = olay.linear(np.abs(xf), np.abs(wg)), olay.linear(np.abs(xf), np.abs(wu))
        tol = 2.0 ** -8 * np.abs(ref) + 2.0 ** -16 * (sg * np.abs(u) + su * np.abs(g / (1 + np.exp(-g))))
        return ref, tol
    wf = to_f32(w).astype(np.float64)
    ref = olay.linear(xf, wf)
    if epi == RES:
        ref = ref + to_f32(res[rows]).astype(np.float64)
    tol = 2.0 ** -8 * np.abs(ref) + 2.0 ** -17 * olay.linear(np.abs(xf), np.abs(wf))
    return ref, tol


def run(torch, m, n, k, epi, x, w_dev_bits, res, in_place=False):
    from paper_2606_05933_amd import ssa
    xd = dev_bf16(torch, x)
    wd = dev_bf16(torch, w_dev_bits)
    nout = n // 2 if epi == SWIGLU else n
    ws_bytes = ssa.linear_workspace_size(m, n, k)
    ws = torch.zeros(max(ws_bytes, 4), dtype=torch.uint8, device="cuda")
    outs = []
    for _ in range(2):
        if in_place:
            out = dev_bf16(torch, res)
            ssa.linear(xd, wd, out, epi, residual=out, workspace=ws)
        else:
            out = torch.full((m, nout), float("nan"), dtype=torch.bfloat16, device="cuda")
            rd = dev_bf16(torch, res) if res is not None else None
            ssa.linear(xd, wd, out, epi, residual=rd, workspace=ws)
        torch.cuda.synchronize()
        outs.append(out.view(torch.int16).cpu().numpy().view(np.uint16))
    assert np.array_equal(outs[0], outs[1]), "two calls in a row differ"
    if ws_bytes:
        assert int(ws[:256].count_nonzero()) == 0, "split tickets not reset"
    return outs[0], ws_bytes


@pytest.mark.parametrize("case", range(len(CASES)))
def test_linear_matches_the_oracle(torch_dev, case):
    from dense_ref import to_f32
    m, n, k, epi = CASES[case]
    say(f"[gpu linear] M={m} N={n} K={k} epilogue={epi}")
    x, w_ref, w_dev, res = inputs(m, n, k, epi, seed=100 + case)
    got, ws_bytes = run(torch_dev, m, n, k, epi, x, w_dev, res)
    rows = np.arange(m) if m * n * k <= 2 ** 33 else np.unique(
        np.r_[0, m - 1, np.arange(0, m, 127), np.random.default_rng(case).integers(0, m, 24)])
    ref, tol = reference(x, w_ref, res, epi, rows)
    g = to_f32(got[rows]).astype(np.float64)
    err = np.abs(g - ref)
    say(f"    ws={ws_bytes} rows={len(rows)} max_err={err.max():.3e} worst_ratio={(err / tol).max():.3f}")
    assert np.isfinite(g).all()
    assert np.all(err <= tol)


def test_linear_residual_in_place(torch_dev):
    from dense_ref import to_f32
    m, n, k = 200, 512, 1024
    x, w, _, res = inputs(m, n, k, RES, seed=7)
    got, _ = run(torch_dev, m, n, k, RES, x, w, res, in_place=True)
    # each call adds x w^T to the buffer: compare the first call only
    from paper_2606_05933_amd import ssa
    xd, wd, out = dev_bf16(torch_dev, x), dev_bf16(torch_dev, w), dev_bf16(torch_dev, res)
    ws = torch_dev.zeros(max(ssa.linear_workspace_size(m, n, k), 4), dtype=torch_dev.uint8,
                         device="cuda")
    ssa.linear(xd, wd, out, RES, residual=out, workspace=ws)
    torch_dev.cuda.synchronize()
    g = to_f32(out.view(torch_dev.int16).cpu().numpy().view(np.uint16)).astype(np.float64)
    ref, tol = reference(x, w, res, RES, np.arange(m))
    assert np.all(np.abs(g - ref) <= tol)


@pytest.mark.parametrize("m,n,k,epi", [(4096, 6144, 4096, NONE), (2048, 28672, 4096, SWIGLU),
                                       (3000, 4096, 14336, RES),
                                       (2176, 4096, 14336, NONE)])
def test_linear_full_size_sampled_rows(torch_dev, m, n, k, epi):
    from dense_ref import to_f32
    say(f"[gpu linear full] M={m} N={n} K={k} epilogue={epi}")
    x, w_ref, w_dev, res = inputs(m, n, k, epi, seed=m + n)
    got, _ = run(torch_dev, m, n, k, epi, x, w_dev, res)
    rows = np.unique(np.r_[0, m - 1, 127, 128, np.random.default_rng(m).integers(0, m, 20)])
    ref, tol = reference(x, w_ref, res, epi, rows)
    err = np.abs(to_f32(got[rows]).astype(np.float64) - ref)
    say(f"    max_err={err.max():.3e} worst_ratio={(err / tol).max():.3f}")
    assert np.all(err <= tol)


def test_linear_rejects_bad_sizes_and_small_workspace(torch_dev):
    from paper_2606_05933_amd import ssa
    torch = torch_dev
    x = torch.zeros((28, 4096), dtype=torch.bfloat16, device="cuda")
    w = torch.zeros((6144, 4096), dtype=torch.bfloat16, device="cuda")
    out = torch.zeros((28, 6144), dtype=torch.bfloat16, device="cuda")
    need = ssa.linear_workspace_size(28, 6144, 4096)
    assert need > 0
    small = torch.zeros(need - 256, dtype=torch.uint8, device="cuda")
    with pytest.raises(ssa.SsaError):
        ssa.linear(x, w, out, NONE, workspace=small)
    with pytest.raises(ssa.SsaError):  # K % 64 != 0
        ssa.linear(x[:, :4000].contiguous(), w[:, :4000].contiguous(), out, NONE)


@pytest.mark.parametrize("m,n", [(1, 8), (37, 4096), (300, 5120), (5, 8192)])
def test_rms_norm_matches_the_oracle(torch_dev, m, n):
    from dense_ref import to_f32
    from oracle import layer as olay
    from paper_2606_05933_amd import ssa, workload
    torch = torch_dev
    say(f"[gpu rms_norm] M={m} N={n}")
    x = workload.normal_bf16((m, n), m + n)
    scale = np.where(np.arange(m) % 3 == 1, 100.0, np.where(np.arange(m) % 3 == 2, 1e-3, 1.0))
    xs = workload.f32_to_bf16_bits(to_f32(x) * scale[:, None].astype(np.float32))
    wt = workload.normal_bf16((n,), 5)
    out = torch.full((m, n), float("nan"), dtype=torch.bfloat16, device="cuda")
    ssa.rms_norm(dev_bf16(torch, xs), dev_bf16(torch, wt), out, eps=1e-5)
    torch.cuda.synchronize()
    g = to_f32(out.view(torch.int16).cpu().numpy().view(np.uint16)).astype(np.float64)
    xf, wf = to_f32(xs).astype(np.float64), to_f32(wt).astype(np.float64)
    ref = olay.rms_norm(xf, wf, eps=1e-5)
    rms = np.sqrt(np.mean(xf * xf, axis=1, keepdims=True) + 1e-5)
    tol = 2.0 ** -8 * np.abs(ref) + 2.0 ** -20 * np.abs(xf * wf) / rms
    assert np.all(np.abs(g - ref) <= tol)
