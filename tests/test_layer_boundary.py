"""Host-side checks of the layer entry points (include/ssa_layer.h): argument
validation happens before any HIP call, so it runs without a GPU; the split-K
workspace rule.  No GPU."""
import ctypes

import pytest

from paper_2606_05933_amd import ssa

LIB = ssa.LIB
NULL = ctypes.c_void_p(None)


def ws(m, n, k):
    out = ctypes.c_size_t(0)
    rc = LIB.ssa_linear_workspace_size(m, n, k, ctypes.byref(out))
    return rc, out.value


@pytest.mark.parametrize("m,n,k", [(-1, 128, 64), (4, 100, 64), (4, 128, 65), (4, 0, 64),
                                   (4, 128, 0), (2 ** 31 - 1, 1 << 20, 64)])
def test_linear_rejects_bad_sizes(m, n, k):
    assert ws(m, n, k)[0] == ssa.SSA_ERR_ARG
    assert LIB.ssa_linear(m, n, k, 0, NULL, NULL, NULL, NULL, NULL, 0, NULL) == ssa.SSA_ERR_ARG


def test_linear_rejects_a_bad_epilogue_and_null_pointers():
    assert LIB.ssa_linear(4, 128, 64, 3, NULL, NULL, NULL, NULL, NULL, 0, NULL) == ssa.SSA_ERR_ARG
    assert LIB.ssa_linear(4, 128, 64, 0, NULL, NULL, NULL, NULL, NULL, 0, NULL) == ssa.SSA_ERR_NULL
    # an empty product needs no pointers
    assert LIB.ssa_linear(0, 128, 64, 0, NULL, NULL, NULL, NULL, NULL, 0, NULL) == ssa.SSA_OK


def test_linear_workspace_rule():
    # enough 128 x 128 tiles to fill the chip: one pass over K, no workspace
    assert ws(2048, 4096, 4096) == (0, 0)
    assert ws(0, 4096, 4096) == (0, 0)
    # a decode-only batch: few tiles, K split; tickets (256 B) + fp32 partial
    # tiles, at most one per 256 of K for each of the M x N outputs' tiles
    rc, b = ws(28, 6144, 4096)
    assert rc == 0 and b > 256 and (b - 256) % (4 * 6144) == 0
    assert b - 256 <= 4 * 6144 * 256 * (4096 // 256)


def test_rms_norm_rejects_bad_arguments():
    f = ctypes.c_float
    assert LIB.ssa_rms_norm(4, 12, NULL, NULL, f(1e-5), NULL, NULL) == ssa.SSA_ERR_ARG
    assert LIB.ssa_rms_norm(4, 8200, NULL, NULL, f(1e-5), NULL, NULL) == ssa.SSA_ERR_ARG
    assert LIB.ssa_rms_norm(4, 64, NULL, NULL, f(-1.0), NULL, NULL) == ssa.SSA_ERR_ARG
    assert LIB.ssa_rms_norm(4, 64, NULL, NULL, f(float("nan")), NULL, NULL) == ssa.SSA_ERR_ARG
    assert LIB.ssa_rms_norm(4, 64, NULL, NULL, f(1e-5), NULL, NULL) == ssa.SSA_ERR_NULL
    assert LIB.ssa_rms_norm(0, 64, NULL, NULL, f(1e-5), NULL, NULL) == ssa.SSA_OK
