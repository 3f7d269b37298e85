"""Test-side helpers, independent of both the oracle and the library.

* ``dense_attention``: brute-force causal softmax attention in numpy fp64 over
  contiguous (unpaged) per-request sequences - the textbook definition.
* ``page_out``: scatter contiguous per-request sequences into the paged pools
  (key page [P, D] slot-major, value page [D, P] dim-major) with its own index
  arithmetic, poisoning every slot it does not fill.
* ``gather``: read a request's sequence back out of the pools.
"""
import numpy as np

NAN16 = np.uint16(0x7FC0)


def to_f32(bits):
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def to_bf16(x):
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    return ((u + (((u >> 16) & 1) + 0x7FFF)) >> 16).astype(np.uint16)


def dense_attention(q, k, v, u, scale):
    """q [c, Hq, D], k/v [u+c, Hkv, D] (float64).  Row j attends keys 0..u+j."""
    c, hq, d = q.shape
    hkv = k.shape[1]
    g = hq // hkv
    out = np.zeros((c, hq, d))
    pos = u + np.arange(c)
    keys = np.arange(k.shape[0])
    mask = keys[None, :] <= pos[:, None]
    for h in range(hq):
        kk = k[:, h // g, :]
        vv = v[:, h // g, :]
        s = scale * (q[:, h, :] @ kk.T)
        s = np.where(mask, s, -np.inf)
        s = s - s.max(axis=1, keepdims=True)
        w = np.exp(s)
        w = w / w.sum(axis=1, keepdims=True)
        out[:, h, :] = w @ vv
    return out


def page_out(seqs_k, seqs_v, hkv, d, P, rng, spare=5, maxp_extra=0):
    """seqs_*: list of uint16 arrays [L_i, Hkv, D].  Returns block_table, kc, vc."""
    lens = [s.shape[0] for s in seqs_k]
    need = [(L + P - 1) // P for L in lens]
    npages = sum(need) + spare
    perm = rng.permutation(npages)
    maxp = max(1, max(need) if need else 1) + maxp_extra
    bt = np.full((len(lens), maxp), -1, dtype=np.int32)
    kc = np.full((npages, hkv, P, d), NAN16, dtype=np.uint16)
    vc = np.full((npages, hkv, d, P), NAN16, dtype=np.uint16)
    o = 0
    for i, L in enumerate(lens):
        bt[i, :need[i]] = perm[o:o + need[i]]
        o += need[i]
        for t in range(L):
            pg, sl = bt[i, t // P], t % P
            kc[pg, :, sl, :] = seqs_k[i][t]
            vc[pg, :, :, sl] = seqs_v[i][t]
    return bt, kc, vc


def gather(kc, vc, bt_row, L, P):
    hkv, d = kc.shape[1], kc.shape[3]
    k = np.zeros((L, hkv, d), dtype=np.uint16)
    v = np.zeros((L, hkv, d), dtype=np.uint16)
    for t in range(L):
        pg, sl = bt_row[t // P], t % P
        k[t] = kc[pg, :, sl, :]
        v[t] = vc[pg, :, :, sl]
    return k, v
