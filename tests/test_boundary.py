"""Host-side tests of the C ABI (no GPU): exports, argument validation, and the
plan's coverage of the batch (SlidingServe Sec. 3.2: B = {(c_i, u_i)}, Eq. 2
routing, Eq. 3 scene, Tab. 1 features)."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2606_05933_amd import ssa, workload

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

HDR = np.dtype([("magic", "<u4"), ("version", "<u4"), ("hash", "<u8"), ("num_reqs", "<i4"),
                ("num_tokens", "<i4"), ("num_items", "<i4"), ("num_chunk_items", "<i4"),
                ("num_decode_items", "<i4"), ("num_groups", "<i4"), ("num_segments", "<i4"),
                ("hq", "<i4"), ("hkv", "<i4"), ("head_dim", "<i4"), ("page_size", "<i4"),
                ("max_pages_per_req", "<i4"), ("num_pages", "<i4"), ("chunk_tile_cols", "<i4"),
                ("off_reqs", "<i4"), ("off_items", "<i4"), ("off_groups", "<i4"),
                ("off_segments", "<i4"), ("ws_partials_off", "<i8"), ("ws_bytes", "<i8"),
                ("plan_bytes", "<i8"), ("scale", "<f4"), ("num_chunk_segments", "<i4"),
                ("reserved", "<i4", 2)])
REQ = np.dtype([("q_start", "<i4"), ("q_len", "<i4"), ("ctx_len", "<i4"), ("n_pages", "<i4")])
ITEM = np.dtype([("kind", "<i4"), ("req", "<i4"), ("kvh", "<i4"), ("col0", "<i4"),
                 ("ncols", "<i4"), ("key0", "<i4"), ("key1", "<i4"), ("group", "<i4"),
                 ("split", "<i4"), ("q_start", "<i4"), ("ctx_len", "<i4"), ("nvalid", "<i4")])
GROUP = np.dtype([("nsplit", "<i4"), ("ncols", "<i4"), ("ws_off", "<i8")])
SEG = np.dtype([("req", "<i4"), ("row0", "<i4"), ("pos0", "<i4"), ("n", "<i4")])


def parse(blob):
    blob = np.asarray(blob, dtype=np.uint8)
    h = np.frombuffer(blob[:128].tobytes(), HDR)[0]

    def arr(off, dt, n):
        return np.frombuffer(blob[off: off + dt.itemsize * n].tobytes(), dt)

    return (h, arr(h["off_reqs"], REQ, h["num_reqs"]), arr(h["off_items"], ITEM, h["num_items"]),
            arr(h["off_groups"], GROUP, h["num_groups"]),
            arr(h["off_segments"], SEG, h["num_segments"]))


def shape_of(hq, hkv, d, q_len, ctx_len, extra_pages=0, num_pages=None, scale=None):
    maxp = max([1] + [(u + c + 15) // 16 for c, u in zip(q_len, ctx_len)]) + extra_pages
    npages = num_pages if num_pages is not None else 4096
    return ssa.make_shape(hq, hkv, d, npages, maxp, scale if scale is not None else d ** -0.5)


def test_library_exports_every_declared_symbol():
    declared = set()
    for h in sorted(os.listdir(os.path.join(ROOT, "include"))):
        if h.endswith(".h"):
            text = open(os.path.join(ROOT, "include", h)).read()
            declared |= set(re.findall(r"\b(ssa_[a-z0-9_]+)\s*\(", text))
    assert declared == set(ssa.EXPORTED)
    lib = ctypes.CDLL(ssa.LIB_PATH)
    for name in declared:
        assert hasattr(lib, name), name


def check_plan_covers_batch(hq, hkv, d, q_len, ctx_len, tuning=None):
    shape = shape_of(hq, hkv, d, q_len, ctx_len)
    blob, info = ssa.ssa_plan(shape, q_len, ctx_len, tuning)
    h, reqs, items, groups, segs = parse(blob)
    G = hq // hkv
    n = len(q_len)
    assert h["magic"] == 0x31415353 and h["num_reqs"] == n
    qs = np.concatenate([[0], np.cumsum(q_len)[:-1]]) if n else np.zeros(0)
    assert np.array_equal(reqs["q_start"], qs) and np.array_equal(reqs["q_len"], q_len)
    # every (row, head) is covered by key ranges that partition [0, pos + 1)
    cover = {}
    for it in items:
        i = it["req"]
        c, u = int(q_len[i]), int(ctx_len[i])
        assert (it["q_start"], it["ctx_len"], it["nvalid"]) == (int(reqs["q_start"][i]), u, u + c)
        if it["kind"] == 1:
            assert c == 1 and it["ncols"] == G
            cols = [(int(reqs["q_start"][i]), it["kvh"] * G + hg, u) for hg in range(G)]
        else:
            assert c > 1
            cols = []
            for cc in range(it["col0"], it["col0"] + it["ncols"]):
                j, hg = divmod(cc, G)
                assert j < c
                cols.append((int(reqs["q_start"][i]) + j, it["kvh"] * G + hg, u + j))
        for row, head, pos in cols:
            lo, hi = it["key0"], min(it["key1"], pos + 1)
            if hi > lo:
                cover.setdefault((row, head), []).append((lo, hi))
            else:  # a split beyond this column's diagonal: empty but allowed
                assert it["group"] >= 0
    for i in range(n):
        for j in range(int(q_len[i])):
            for head in range(hq):
                rngs = sorted(cover.pop((int(reqs["q_start"][i]) + j, head)))
                assert rngs[0][0] == 0 and rngs[-1][1] == int(ctx_len[i]) + j + 1
                assert all(a[1] == b[0] for a, b in zip(rngs, rngs[1:]))
    assert not cover
    # merge groups: every split exactly once, records disjoint and inside the workspace
    for gi, g in enumerate(groups):
        mem = items[items["group"] == gi]
        assert sorted(mem["split"]) == list(range(g["nsplit"]))
        assert (mem["ncols"] == g["ncols"]).all()
        end = h["ws_partials_off"] + 4 * (g["ws_off"] + g["nsplit"] * g["ncols"] * (d + 2))
        assert end <= h["ws_bytes"]
    offs = sorted((g["ws_off"], g["ws_off"] + g["nsplit"] * g["ncols"] * (d + 2)) for g in groups)
    assert all(a[1] <= b[0] for a, b in zip(offs, offs[1:]))
    assert ((items["group"] < 0) | (items["group"] < len(groups))).all()
    # append segments: each new token exactly once, inside one page
    seen = []
    for sg in segs:
        assert sg["pos0"] // 16 == (sg["pos0"] + sg["n"] - 1) // 16
        i = sg["req"]
        for k in range(sg["n"]):
            seen.append((sg["row0"] + k, sg["pos0"] + k - int(ctx_len[i])))
    expect = [(int(reqs["q_start"][i]) + j, j) for i in range(n) for j in range(int(q_len[i]))]
    assert sorted(seen) == sorted(expect)
    # those of chunk requests (c > 1) first, then one per decode request
    nc, ql = int(h["num_chunk_segments"]), np.asarray(q_len)
    assert (ql[segs["req"][:nc]] > 1).all() and (ql[segs["req"][nc:]] == 1).all()
    assert len(segs) - nc == int((ql == 1).sum())
    return info, items


PLAN_CASES = [
    (8, 8, 64, [64, 1, 1, 1, 1], [192, 128, 256, 384, 512]),
    (32, 8, 128, [512] + [1] * 9, [2048] + list(range(500, 4100, 400))),
    (28, 4, 128, [64, 256, 0, 1, 1, 3], [7000, 13, 5, 0, 16383, 1]),
    (16, 16, 64, [2, 1, 0], [0, 0, 0]),
    (4, 1, 128, [1000, 1], [33000, 32767]),
]


@pytest.mark.parametrize("case", PLAN_CASES)
def test_plan_partitions_every_output_key_range(case):
    hq, hkv, d, q_len, ctx_len = case
    check_plan_covers_batch(hq, hkv, d, np.array(q_len, np.int32), np.array(ctx_len, np.int32))


@pytest.mark.parametrize("tile", [32, 64, 128])
@pytest.mark.parametrize("csplit", [0, 1024, 4096])
def test_plan_partitions_under_tuning(tile, csplit):
    q_len = np.array([700, 33, 1, 1], np.int32)
    ctx_len = np.array([5000, 100, 9000, 31], np.int32)
    tu = ssa.make_tuning(chunk_tile_cols=tile, chunk_split_keys=csplit, decode_split_keys=512)
    info, items = check_plan_covers_batch(28, 4, 128, q_len, ctx_len, tu)
    assert info.num_items == len(items)


@pytest.mark.parametrize("order", [1, 2, 3, 4])
@pytest.mark.parametrize("cus", [4, 256])
def test_plan_partitions_under_every_launch_order(order, cus):
    shape, q_len, ctx_len = workload.workload_lengths("multi", seed=5)
    tu = ssa.make_tuning(mix_order=order, num_cus=cus)
    info, items = check_plan_covers_batch(shape.hq, shape.hkv, shape.d, q_len, ctx_len, tu)
    is_chunk = items["kind"] == 0
    nc, nd = int(is_chunk.sum()), int((~is_chunk).sum())
    assert nc > 0 and nd > 0
    if order == 1:  # all chunk items first
        assert is_chunk[:nc].all()
    if order in (3, 4):  # min(cus, chunk items) chunk items, then decode items up to 2 * cus
        first = min(cus, nc)
        second = min(nd, 2 * cus - first)
        assert is_chunk[:first].all()
        assert not is_chunk[first:first + second].any()
    if order == 4:  # then every other decode item, then the other chunk items
        assert not is_chunk[first:first + nd].any()
        assert is_chunk[first + nd:].all()


def test_plan_on_generated_workloads():
    for name in workload.WORKLOADS:
        shape, q_len, ctx_len = workload.workload_lengths(name, seed=3)
        check_plan_covers_batch(shape.hq, shape.hkv, shape.d, q_len, ctx_len)


def test_scene_and_features_follow_the_paper():
    # Eq. 2: D = {c <= 1}, P = {c > 1}; Eq. 3 scene; Tab. 1 features x1..x7
    q_len = np.array([5, 1, 0, 9, 1], np.int32)
    ctx_len = np.array([10, 20, 30, 0, 7], np.int32)
    shape = shape_of(8, 2, 64, q_len, ctx_len)
    _, info = ssa.ssa_plan(shape, q_len, ctx_len)
    # a request with no new token (c = 0) runs nothing: it is in no feature
    P = q_len > 1
    Dm = q_len == 1
    B = q_len > 0
    x = [np.sum(q_len[P] * (ctx_len[P] + q_len[P])), np.sum(q_len[P] ** 2), np.sum(ctx_len[B]),
         np.sum(Dm), np.sum(ctx_len[Dm]), np.sum(q_len[P]), np.max(q_len[P])]
    assert list(info.x) == [float(v) for v in x]
    assert info.scene == 3 and info.num_decode_reqs == 2 and info.num_chunk_reqs == 2
    hq, hkv, d = 8, 2, 64
    cf = sum(4 * hq * d * (c * u + c * (c + 1) / 2) for c, u in zip(q_len[P], ctx_len[P]))
    assert info.chunk_flops == cf
    db = sum((u + 1) * hkv * d * 4 + 2 * hq * d * 2 for c, u in zip(q_len, ctx_len) if c == 1)
    assert info.decode_bytes == db
    for ql, scene in (([1, 1, 0], 1), ([4, 2], 2), ([0, 0], 0), ([], 0), ([4, 0], 2)):
        ql = np.array(ql, np.int32)
        cl = np.zeros_like(ql)
        _, inf = ssa.ssa_plan(shape_of(8, 2, 64, ql, cl), ql, cl)
        assert inf.scene == scene


def _lengths_plan(name, chunk, tuning=None, keep=None):
    """Plan (blob, info) of a named workload's lengths (no tensors drawn);
    keep: optional filter on q_len (e.g. the chunk rows alone)."""
    from paper_2606_05933_amd import workload
    s, q_len, ctx_len = workload.workload_lengths(name, 0, chunk)
    q_len, ctx_len = np.asarray(q_len, np.int32), np.asarray(ctx_len, np.int32)
    if keep is not None:
        m = keep(q_len)
        q_len, ctx_len = q_len[m], ctx_len[m]
    pages = int(sum((u + c + 15) // 16 for c, u in zip(q_len, ctx_len)))
    shape = shape_of(s.hq, s.hkv, s.d, q_len, ctx_len, num_pages=pages + 64)
    return ssa.ssa_plan(shape, q_len, ctx_len, tuning)


def _plan_kinds(name, chunk, tuning=None):
    """Work-item kinds of a generated workload's plan, in launch order."""
    blob, info = _lengths_plan(name, chunk, tuning)
    hdr = np.frombuffer(blob[:128].tobytes(), dtype=np.int32)
    off = int(hdr[19])  # off_items
    items = np.frombuffer(blob[off:off + 48 * info.num_items].tobytes(), np.int32).reshape(-1, 12)
    return items[:, 0], info


def test_automatic_launch_order_pairs_only_decode_heavy_full_chunk_batches():
    """Left at 0, mix_order pairs chunk and decode items on every unit when the chunk
    items fill both slots of every unit and the decode part is comparable (l8b at
    c = 2048); with a smaller decode part (l70b at c = 1024) the other decode items
    follow the pairs and the other chunk items come last; batches with fewer chunk
    items (l8b at c = 512) keep all chunk items first; an explicit order is kept."""
    def paired(kinds, info):
        # paired: the first 256 workgroups are chunk items, the next 256 decode items
        return bool(info.num_chunk_items >= 512 and (kinds[256:512] != kinds[0]).all()
                    and (kinds[:256] == kinds[0]).all())
    k, info = _plan_kinds("l8b", 2048)
    assert paired(k, info)
    k, info = _plan_kinds("l8b", 2048, ssa.make_tuning(mix_order=1))
    assert not paired(k, info) and (k[:512] == k[0]).all()
    # chunk-heavy with a sizeable decode part (l70b at c = 1024, estimated ratio
    # 0.56): one chunk item per unit beside the decode items, the decode items
    # next, the other chunk items last
    k, info = _plan_kinds("l70b", 1024)
    assert info.num_chunk_items == 512 and paired(k, info)
    assert (k[512:512 + info.num_decode_items - 256] == 1).all() and (k[-256:] == 0).all()
    k, info = _plan_kinds("l8b", 512)
    assert (k[:info.num_chunk_items] == k[0]).all()  # all chunk items first


def test_automatic_chunk_splits_fill_the_last_round():
    """With the split length left at 0, chunk tiles that would leave the last
    round of the 512 workgroup slots part empty are cut: the 70B-shaped chunk of
    1536 tokens alone (768 tiles) runs as 1536 pieces (three rounds of half
    tiles), while 512 tiles (c = 1024) and 1024 tiles (c = 2048), whole rounds,
    stay whole; an explicit split length is kept."""
    chunk_rows = lambda q: q > 1
    for chunk, items in ((1024, 512), (1536, 1536), (2048, 1024)):
        _, info = _lengths_plan("l70b", chunk, keep=chunk_rows)
        assert info.num_chunk_items == items, (chunk, info.num_chunk_items)
        _, info = _lengths_plan("l70b", chunk, ssa.make_tuning(chunk_split_keys=1 << 20),
                                keep=chunk_rows)
        assert info.num_chunk_items == 768 * chunk // 1536, chunk


def test_plan_is_deterministic():
    q_len = np.array([300, 1, 1, 1], np.int32)
    ctx_len = np.array([0, 5, 900, 40], np.int32)
    shape = shape_of(32, 8, 128, q_len, ctx_len)
    a, _ = ssa.ssa_plan(shape, q_len, ctx_len)
    b, _ = ssa.ssa_plan(shape, q_len, ctx_len)
    assert a.tobytes() == b.tobytes()
    c, _ = ssa.ssa_plan(shape, q_len, ctx_len + np.array([0, 0, 1, 0], np.int32))
    assert parse(a)[0]["hash"] != parse(c)[0]["hash"]


# ---------------------------------------------------------------- validation

def plan_rc(shape, q_len, ctx_len, tuning=None, cap=None):
    ql = np.asarray(q_len, np.int32)
    cl = np.asarray(ctx_len, np.int32)
    buf = np.zeros(cap if cap is not None else 1 << 16, np.uint8)
    info = ssa.SsaPlanInfo()
    return ssa.LIB.ssa_plan(ctypes.byref(shape), ql.ctypes.data if ql.size else None,
                            cl.ctypes.data if cl.size else None, ql.shape[0],
                            ctypes.byref(tuning) if tuning is not None else None,
                            buf.ctypes.data, buf.nbytes, ctypes.byref(info)), buf


@pytest.mark.parametrize("mutate,code", [
    (dict(num_q_heads=0), -2), (dict(num_kv_heads=3), -2), (dict(num_q_heads=34, num_kv_heads=2), -2),
    (dict(head_dim=96), -3), (dict(page_size=8), -4), (dict(softmax_scale=float("inf")), -11),
    (dict(softmax_scale=-0.5), -11),
    (dict(num_pages=0), -6), (dict(max_pages_per_req=0), -6),
])
def test_bad_shape_codes(mutate, code):
    shape = ssa.make_shape(8, 2, 64, 100, 8, 0.125)
    for k, v in mutate.items():
        setattr(shape, k, v)
    rc, buf = plan_rc(shape, [3, 1], [5, 6])
    assert rc == code
    assert not buf.any()  # nothing written on error
    assert ssa.ssa_status_string(code) not in ("ok", "unknown")


def test_bad_lengths_and_pages_and_buffers():
    shape = ssa.make_shape(8, 2, 64, 100, 4, 0.125)
    assert plan_rc(shape, [-1, 1], [5, 6])[0] == -5
    assert plan_rc(shape, [1, 1], [5, -6])[0] == -5
    assert plan_rc(shape, [1, 1], [5, 64])[0] == -6  # 65 keys need 5 pages > 4
    assert plan_rc(shape, [1, 1], [5, 63])[0] == 0
    assert plan_rc(shape, [1, 1], [5, 6], cap=64)[0] == -7
    assert plan_rc(shape, [1], [5], tuning=ssa.make_tuning(chunk_tile_cols=96))[0] == -12
    assert plan_rc(shape, [1], [5], tuning=ssa.make_tuning(decode_split_keys=100))[0] == -12
    pb, wb = ctypes.c_size_t(), ctypes.c_size_t()
    assert ssa.LIB.ssa_plan_size(None, None, None, 0, None, ctypes.byref(pb), ctypes.byref(wb)) == -1
    assert ssa.LIB.ssa_plan_size(ctypes.byref(shape), None, None, 2, None, ctypes.byref(pb),
                                 ctypes.byref(wb)) == -1
    assert ssa.ssa_status_string(12345) == "unknown"


def test_launchers_validate_before_any_hip_call():
    q_len = np.array([40, 1, 1], np.int32)
    ctx_len = np.array([5000, 3000, 9000], np.int32)
    shape = shape_of(32, 8, 128, q_len, ctx_len)
    blob, info = ssa.ssa_plan(shape, q_len, ctx_len, ssa.make_tuning(decode_split_keys=1024))
    assert info.num_merge_groups > 0
    fake = ctypes.c_void_p(0x1000)  # never dereferenced: every call below fails validation
    L = ssa.LIB
    p = blob.ctypes.data
    # NULL arguments
    assert L.ssa_kv_append(ctypes.byref(shape), p, None, fake, fake, fake, fake, fake, None) == -1
    assert L.ssa_kv_append(ctypes.byref(shape), p, fake, None, fake, fake, fake, fake, None) == -1
    assert L.ssa_mixed_attention(ctypes.byref(shape), p, fake, fake, fake, fake, fake, None, fake,
                                 1 << 30, None) == -1
    assert L.ssa_mixed_attention(ctypes.byref(shape), None, fake, fake, fake, fake, fake, fake,
                                 fake, 1 << 30, None) == -1
    # workspace too small / missing
    _, ws = ssa.ssa_plan_size(shape, q_len, ctx_len, ssa.make_tuning(decode_split_keys=1024))
    assert ws > 0
    assert L.ssa_mixed_attention(ctypes.byref(shape), p, fake, fake, fake, fake, fake, fake, fake,
                                 ws - 1, None) == -8
    assert L.ssa_mixed_attention(ctypes.byref(shape), p, fake, fake, fake, fake, fake, fake, None,
                                 ws, None) == -8
    # a plan of another shape
    other = shape_of(32, 8, 128, q_len, ctx_len, num_pages=77)
    assert L.ssa_mixed_attention(ctypes.byref(other), p, fake, fake, fake, fake, fake, fake, fake,
                                 ws, None) == -9
    assert L.ssa_kv_append(ctypes.byref(other), p, fake, fake, fake, fake, fake, fake, None) == -9
    junk = np.zeros(256, np.uint8)
    assert L.ssa_kv_append(ctypes.byref(shape), junk.ctypes.data, fake, fake, fake, fake, fake,
                           fake, None) == -9
    # the timed entry points validate the same way (events are never touched)
    assert L.ssa_kv_append_timed(ctypes.byref(shape), p, None, fake, fake, fake, fake, fake, None,
                                 fake, fake) == -1
    assert L.ssa_kv_append_timed(ctypes.byref(other), p, fake, fake, fake, fake, fake, fake, None,
                                 fake, fake) == -9
    assert L.ssa_mixed_attention_timed(ctypes.byref(shape), p, fake, fake, fake, fake, fake, fake,
                                       fake, ws - 1, None, fake, fake) == -8
    assert L.ssa_mixed_attention_timed(ctypes.byref(other), p, fake, fake, fake, fake, fake, fake,
                                       fake, ws, None, fake, fake) == -9
    # kv_append + attention in one launch: the same checks
    args = [fake] * 8  # q, k_new, v_new, k_cache, v_cache, block_table, out, workspace
    assert L.ssa_append_attention(ctypes.byref(shape), p, None, *args, ws, None, None, None) == -1
    assert L.ssa_append_attention(ctypes.byref(other), p, fake, *args, ws, None, None, None) == -9
    assert L.ssa_append_attention(ctypes.byref(shape), p, fake, *args, ws - 1, None, None,
                                  None) == -8
    nulls = list(args)
    nulls[1] = None  # k_new
    assert L.ssa_append_attention(ctypes.byref(shape), p, fake, *nulls, ws, None, None, None) == -1
    nulls = list(args)
    nulls[7] = None  # workspace
    assert L.ssa_append_attention(ctypes.byref(shape), p, fake, *nulls, ws, None, None, None) == -8
    # In a fused launch the last chunk item resets the counters, so a plan whose chunk
    # requests have append segments must have chunk items.  A header that says it has none
    # still passes the plan check (the attention call gets as far as its workspace) but is
    # refused by the fused call.
    bad = blob.copy()
    hdr = bad[:128].view(np.int32)  # int32 7: num_chunk_items
    assert hdr[7] > 0
    hdr[7] = 0
    q = bad.ctypes.data
    assert L.ssa_mixed_attention(ctypes.byref(shape), q, fake, fake, fake, fake, fake, fake, fake,
                                 ws - 1, None) == -8
    assert L.ssa_append_attention(ctypes.byref(shape), q, fake, *args, ws, None, None, None) == -9


def test_streams_launcher_validates_before_any_hip_call():
    """ssa_append_attention_streams checks what ssa_append_attention checks, in
    every launch order, before any HIP call."""
    q_len = np.array([40, 1, 1, 64], np.int32)
    ctx_len = np.array([5000, 3000, 9000, 100], np.int32)
    shape = shape_of(32, 8, 128, q_len, ctx_len)
    fake = ctypes.c_void_p(0x1000)  # never dereferenced: every call below fails validation
    L = ssa.LIB
    args = [fake] * 8  # q, k_new, v_new, k_cache, v_cache, block_table, out, workspace
    other = shape_of(32, 8, 128, q_len, ctx_len, num_pages=77)
    for order in range(7):
        tu = ssa.make_tuning(decode_split_keys=1024, mix_order=order, num_cus=4)
        blob, info = ssa.ssa_plan(shape, q_len, ctx_len, tu)
        _, ws = ssa.ssa_plan_size(shape, q_len, ctx_len, tu)
        p = blob.ctypes.data
        assert L.ssa_append_attention_streams(ctypes.byref(shape), p, None, *args, ws, None,
                                              fake, None, None) == -1
        assert L.ssa_append_attention_streams(ctypes.byref(other), p, fake, *args, ws, None,
                                              fake, None, None) == -9
        assert L.ssa_append_attention_streams(ctypes.byref(shape), p, fake, *args, ws - 1, None,
                                              fake, None, None) == -8
        nulls = list(args)
        nulls[1] = None  # k_new
        assert L.ssa_append_attention_streams(ctypes.byref(shape), p, fake, *nulls, ws, None,
                                              fake, None, None) == -1
    assert plan_rc(shape, q_len, ctx_len, tuning=ssa.make_tuning(mix_order=7))[0] == -12


def _streams_split(name, chunk=None, tuning=None):
    shape, q_len, ctx_len = workload.workload_lengths(name, seed=0, chunk=chunk)
    s = ssa.make_shape(shape.hq, shape.hkv, shape.d, 1 << 20, 4096, shape.softmax_scale)
    blob, info = ssa.ssa_plan(s, q_len, ctx_len, tuning)
    h, _, items, _, _ = parse(blob)
    return int(h["reserved"][1]), items["kind"], info


def test_plan_records_the_two_stream_split():
    """The plan's streams_beside field: -1 (one launch) unless mix_order asks for
    the two-stream launch.  Order 5 splits where the chunk items fill both slots
    of every unit in one round and the decode bytes fit beside the chunk rows
    (the 70B-shaped batch at c = 1024: every decode item beside), with chunk
    items first; elsewhere it keeps the automatic one-launch order and -1.
    Order 6 always splits, half of the decode items beside."""
    for order in (0, 1, 2, 3, 4):
        beside, _, _ = _streams_split("l70b", tuning=ssa.make_tuning(mix_order=order))
        assert beside == -1
    beside, kinds, info = _streams_split("l70b", None, ssa.make_tuning(mix_order=5))
    nc = info.num_chunk_items
    assert nc == 512 and (kinds[:nc] == 0).all() and (kinds[nc:] == 1).all()
    assert beside == info.num_decode_items
    # two rounds of chunk tiles (c = 2048), fewer than 1.5 per unit (c = 512),
    # or a decode part too large for the chunk rows' time (l8b): one launch, in
    # the automatic order
    for name, chunk in (("l70b", 2048), ("l70b", 512), ("l8b", None), ("l8b", 2048),
                        ("multi", None)):
        beside, kinds, _ = _streams_split(name, chunk, ssa.make_tuning(mix_order=5))
        auto, kinds0, _ = _streams_split(name, chunk, None)
        assert beside == -1 and auto == -1 and np.array_equal(kinds, kinds0), (name, chunk)
    beside, kinds, info = _streams_split("l8b", None, ssa.make_tuning(mix_order=6))
    nc = info.num_chunk_items
    assert (kinds[:nc] == 0).all() and beside == (info.num_decode_items + 1) // 2


def test_block_table_check_covers_exactly_the_entries_the_kernels_read():
    # request 3 has no new token: no work item and no append segment reads its row
    from paper_2606_05933_amd import workload
    q_len = np.array([40, 1, 1, 0], np.int32)
    ctx_len = np.array([5000, 3000, 17, 33], np.int32)
    b = workload.make_batch(workload.Shape(32, 8, 128), q_len, ctx_len, seed=3)
    s = b.shape
    shape = ssa.make_shape(s.hq, s.hkv, s.d, b.num_pages, b.block_table.shape[1], s.softmax_scale)
    blob, _ = ssa.ssa_plan(shape, q_len, ctx_len, None)
    bt = b.block_table.copy()
    ssa.check_block_table(shape, blob, bt)  # the generated table is valid
    need = np.where(q_len > 0, (ctx_len + q_len + 15) // 16, 0)
    for i in range(len(q_len)):
        if need[i] == 0:
            t = bt.copy()
            t[i, :] = -1  # never read
            ssa.check_block_table(shape, blob, t)
            continue
        for bad in (-1, b.num_pages):
            t = bt.copy()
            t[i, need[i] - 1] = bad  # the request's last entry that is read
            with pytest.raises(ssa.SsaError):
                ssa.check_block_table(shape, blob, t)
        if need[i] < bt.shape[1]:
            t = bt.copy()
            t[i, need[i]:] = -7  # entries past the request's pages are never read
            ssa.check_block_table(shape, blob, t)
    assert ssa.LIB.ssa_check_block_table(ctypes.byref(shape), blob.ctypes.data, None) == -1
    # the binding refuses a table whose shape the library would read past
    with pytest.raises(ValueError):
        ssa.check_block_table(shape, blob, bt[:, :-1])
    with pytest.raises(ValueError):
        ssa.check_block_table(shape, blob, bt[:-1])

    other = shape_of(32, 8, 128, q_len, ctx_len, num_pages=b.num_pages + 1)
    assert ssa.LIB.ssa_check_block_table(ctypes.byref(other), blob.ctypes.data,
                                         bt.ctypes.data) == -9


def test_plan_refuses_sizes_beyond_its_int32_fields():
    # 2^27 + 1 chunk tokens at G = 16: 2^31 + 16 columns do not fit the items' int32
    # column fields
    shape = ssa.make_shape(16, 1, 64, 1 << 20, (1 << 27) // 16 + 2, 0.125)
    with pytest.raises(ssa.SsaError) as e:
        ssa.ssa_plan_size(shape, [(1 << 27) + 1], [0])
    assert e.value.code == -5
    # a plan blob beyond 2^31 bytes: tiny decode pieces would make over 2^31 / 48
    # items (refused before they are generated)
    shape = ssa.make_shape(8, 8, 64, 1 << 20, (1 << 28) // 16 + 1, 0.125)
    tun = ssa.make_tuning(decode_split_keys=32)
    with pytest.raises(ssa.SsaError) as e:
        ssa.ssa_plan_size(shape, [1] * 6, [(1 << 28) - 1] * 6, tun)
    assert e.value.code == -5


def test_empty_batch_launches_nothing():
    shape = ssa.make_shape(8, 2, 64, 10, 1, 0.125)
    blob, info = ssa.ssa_plan(shape, np.zeros(0, np.int32), np.zeros(0, np.int32))
    assert info.num_items == 0 and info.scene == 0
    L = ssa.LIB
    # no work: returns OK without touching (NULL) buffers or launching
    assert L.ssa_kv_append(ctypes.byref(shape), blob.ctypes.data, ctypes.c_void_p(0x1000), None,
                           None, None, None, None, None) == 0
    assert L.ssa_mixed_attention(ctypes.byref(shape), blob.ctypes.data, ctypes.c_void_p(0x1000),
                                 None, None, None, None, None, None, 0, None) == 0


def test_generator_is_deterministic_and_poisons_unwritten_slots():
    a = workload.make_workload("tiny", seed=4)
    b = workload.make_workload("tiny", seed=4)
    c = workload.make_workload("tiny", seed=5)
    assert a.digest() == b.digest() != c.digest()
    nan = workload.BF16_NAN
    for i, (cq, u) in enumerate(zip(a.q_len, a.ctx_len)):
        for t in range(u, u + cq):
            pg, sl = a.block_table[i, t // 16], t % 16
            assert (a.k_cache[pg, :, sl, :] == nan).all() and (a.v_cache[pg, :, :, sl] == nan).all()
        if u:
            pg = a.block_table[i, (u - 1) // 16]
            assert not (a.k_cache[pg, :, (u - 1) % 16, :] == nan).any()
    used = set(a.block_table[a.block_table >= 0].tolist())
    spare = [p for p in range(a.num_pages) if p not in used]
    assert len(spare) == 64 and (a.k_cache[spare] == nan).all()
    x = np.float32([1.0, 1.00390625, 1.01171875, -2.5, 3.1415926])
    assert np.array_equal(workload.bf16_bits_to_f32(workload.f32_to_bf16_bits(x)),
                          np.float32([1.0, 1.0, 1.015625, -2.5, 3.140625]))


def _fresh_python(code):
    import subprocess
    import sys
    return subprocess.run([sys.executable, "-c", code], capture_output=True, text=True,
                          timeout=300, cwd=ROOT)


def test_binding_shares_torchs_hip_runtime_whatever_is_imported_first():
    """The binding loaded before anything imported torch still ends up with a
    single HIP runtime in the process (torch's): torch's streams and memory are
    only valid in the runtime that made them."""
    r = _fresh_python("from paper_2606_05933_amd import ssa\n"
                      "import torch\n"
                      "rt = ssa.hip_runtimes_loaded()\n"
                      "print(len(rt), rt)\n"
                      "assert len(rt) == 1, rt\n")
    assert r.returncode == 0, r.stdout + r.stderr


def test_binding_refuses_a_process_with_two_hip_runtimes():
    r = _fresh_python("import ctypes\n"
                      "ctypes.CDLL('paper_2606_05933_amd/libssa.so')\n"
                      "from paper_2606_05933_amd import ssa\n")
    assert r.returncode != 0
    assert "more than one HIP runtime" in r.stderr
