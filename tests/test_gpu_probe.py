"""The probe kernels of include/ssa_probe.h compute what they claim, so that the
rates measured with them count real work: the read probe's per-workgroup XORs
combine to the XOR of every word of the buffer (each byte was loaded), the
gather probe's to the XOR of exactly the chunks its index names, and the MFMA
probe's sum equals the closed form of its MFMA chains."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_dev():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    torch.cuda.set_device(0)
    return torch


@pytest.mark.parametrize("words,wgs", [(4, 1), (1 << 20, 37), ((1 << 22) + 12, 4096)])
def test_hbm_read_probe_reads_every_word(torch_dev, words, wgs):
    from paper_2606_05933_amd import ssa
    torch = torch_dev
    host = np.random.default_rng(words).integers(0, 2 ** 32, size=words, dtype=np.uint64).astype(
        np.uint32)
    src = torch.from_numpy(host.view(np.int32)).cuda()
    out = torch.zeros(wgs, dtype=torch.int32, device="cuda")
    assert ssa.probe_hbm_read(src, out, wgs) == words * 4
    torch.cuda.synchronize()
    got = np.bitwise_xor.reduce(out.cpu().numpy().view(np.uint32))
    assert got == np.bitwise_xor.reduce(host)


@pytest.mark.parametrize("chunk_bytes,n,wgs,pattern", [(4096, 64, 2, 0), (1024, 512, 3, 0),
                                                       (16384, 40, 1, 0), (2048, 24, 8, 0),
                                                       (4096, 64, 2, 1), (4096, 100, 3, 1)])
def test_hbm_gather_probe_reads_the_named_chunks(torch_dev, chunk_bytes, n, wgs, pattern):
    """Every chunk the index names is read once, an out-of-range index reads the
    buffer's last chunk, and a wave whose last step runs past the index re-reads
    the last named chunk: the XOR of the per-workgroup results matches a host
    model of that schedule."""
    from paper_2606_05933_amd import ssa
    torch = torch_dev
    rng = np.random.default_rng(chunk_bytes + n)
    src_chunks = n + 5
    host = rng.integers(0, 2 ** 32, size=src_chunks * chunk_bytes // 4, dtype=np.uint64).astype(
        np.uint32)
    index = rng.permutation(src_chunks)[:n].astype(np.int32)
    index[n // 2] = src_chunks + 100  # clamped to the last chunk of the buffer
    src = torch.from_numpy(host.view(np.int32)).cuda()
    idx = torch.from_numpy(index).cuda()
    out = torch.zeros(wgs, dtype=torch.int32, device="cuda")
    assert ssa.probe_hbm_gather(src, idx, chunk_bytes, out, wgs, pattern=pattern) == n * chunk_bytes
    torch.cuda.synchronize()
    # host model: wave w reads chunks c0 .. c0 + cps - 1 for c0 = w cps, w cps + waves cps, ...
    # (a chunk past the end is chunk n - 1 again)
    cps, waves = 16 // (chunk_bytes // 1024), 4 * wgs
    words = host.reshape(src_chunks, chunk_bytes // 4)
    chunk_xor = np.bitwise_xor.reduce(words, axis=1)
    want = np.uint32(0)
    for w in range(waves):
        for c0 in range(w * cps, n, waves * cps):
            for k in range(cps):
                c = min(c0 + k, n - 1)
                want ^= chunk_xor[min(max(int(index[c]), 0), src_chunks - 1)]
    got = np.bitwise_xor.reduce(out.cpu().numpy().view(np.uint32))
    assert got == want


def test_mfma_probe_matches_the_closed_form(torch_dev):
    from dense_ref import to_bf16, to_f32
    from paper_2606_05933_amd import ssa
    torch = torch_dev
    iters, wgs = 8, 3
    out = torch.zeros(wgs, dtype=torch.float32, device="cuda")
    assert ssa.probe_mfma_bf16(iters, wgs, out) == wgs * 4 * iters * 16 * 16384
    torch.cuda.synchronize()
    # lane l supplies row / column l % 16 of k block l // 16: a[j] = s + 0.01 j with
    # s = 0.125 (l % 8), b[j] = 0.5 - 0.01 j, both rounded to bf16
    j = np.arange(8)
    def bf(x):
        return to_f32(to_bf16(np.asarray(x, np.float32))).astype(np.float64)
    b = bf(0.5 - 0.01 * j)
    d = np.zeros((16, 16))
    for r in range(16):
        for g in range(4):
            a = bf(np.float32(0.125 * ((g * 16 + r) % 8)) + np.float32(0.01) * j.astype(np.float32))
            d[r, :] += np.dot(a, b)  # every column of a k block sees the same b
    want = 4 * 16 * iters * d.sum()  # waves x chains x iterations x all 256 outputs
    got = out.cpu().numpy().astype(np.float64)
    assert np.allclose(got, want, rtol=1e-5)
