"""Value-pool layout conversion (ssa_v_pool_convert): token-major pages
[num_pages, Hkv, 16, D] to the dim-major pages [num_pages, Hkv, D, 16] the
attention kernels read, and back.  Bytes move unchanged, so the check is
bit-exact against a transpose of the same bits; the argument checks run on the
host before any HIP call."""
import ctypes

import numpy as np
import pytest

from paper_2606_05933_amd import ssa

ERR_SHAPE, ERR_HEAD_DIM, ERR_PAGE_SIZE, ERR_PAGES = -2, -3, -4, -6  # include/ssa.h


@pytest.fixture(scope="module")
def cuda0():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    torch.cuda.set_device(0)
    return "cuda:0"


def _shape(hkv, d, pages):
    return ssa.make_shape(hkv, hkv, d, pages, 1, 0.125)


def test_v_pool_convert_rejects_bad_arguments():
    L = ssa.LIB
    s = _shape(2, 128, 4)
    a, b = ctypes.c_void_p(1 << 20), ctypes.c_void_p(1 << 30)  # never dereferenced
    assert L.ssa_v_pool_convert(None, a, b, 1, None) == ssa.SSA_ERR_NULL
    assert L.ssa_v_pool_convert(ctypes.byref(s), None, b, 1, None) == ssa.SSA_ERR_NULL
    assert L.ssa_v_pool_convert(ctypes.byref(s), a, None, 1, None) == ssa.SSA_ERR_NULL
    assert L.ssa_v_pool_convert(ctypes.byref(s), a, b, 2, None) == ssa.SSA_ERR_ARG
    assert L.ssa_v_pool_convert(ctypes.byref(s), ctypes.c_void_p((1 << 20) + 8), b, 1,
                                None) == ssa.SSA_ERR_ARG  # misaligned
    pool = 4 * 2 * 16 * 128 * 2
    assert L.ssa_v_pool_convert(ctypes.byref(s), a, ctypes.c_void_p((1 << 20) + pool - 16), 1,
                                None) == ssa.SSA_ERR_ARG  # overlapping
    assert L.ssa_v_pool_convert(ctypes.byref(s), a, a, 0, None) == ssa.SSA_ERR_ARG  # in place
    for bad, rc in ((_shape(2, 96, 4), ERR_HEAD_DIM), (_shape(2, 128, 0), ERR_PAGES),
                    (ssa.make_shape(2, 2, 128, 4, 1, 0.125, page_size=32), ERR_PAGE_SIZE)):
        assert L.ssa_v_pool_convert(ctypes.byref(bad), a, b, 1, None) == rc
    bad = _shape(2, 128, 4)
    bad.num_kv_heads = 0
    assert L.ssa_v_pool_convert(ctypes.byref(bad), a, b, 1, None) == ERR_SHAPE


@pytest.mark.gpu
@pytest.mark.parametrize("hkv,d,pages", [(8, 128, 37), (1, 128, 37), (2, 64, 5), (3, 64, 1),
                                         (1, 128, 1)])
def test_v_pool_convert_is_the_transpose(cuda0, hkv, d, pages):
    import torch
    rng = np.random.default_rng(hkv * 1000 + d + pages)
    tok = rng.integers(0, 1 << 16, size=(pages, hkv, 16, d), dtype=np.uint16)  # any bit patterns
    src = torch.from_numpy(tok.view(np.int16)).to(cuda0)
    dim = torch.empty_like(src)
    back = torch.full_like(src, -1)
    s = _shape(hkv, d, pages)
    ssa.v_pool_convert(s, src, dim, to_dim_major=True)
    ssa.v_pool_convert(s, dim, back, to_dim_major=False)
    torch.cuda.synchronize()
    got = dim.cpu().numpy().view(np.uint16).reshape(pages, hkv, d, 16)
    assert np.array_equal(got, np.ascontiguousarray(tok.transpose(0, 1, 3, 2)))
    assert np.array_equal(back.cpu().numpy().view(np.uint16), tok)
