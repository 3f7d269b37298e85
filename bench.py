#!/usr/bin/env python3
"""Benchmark of one serving iteration's attention hot path on one MI355X.

A step is the whole path for one batch B = {(c_i, u_i)} (SlidingServe Sec. 3.2):
host planning (routing by Eq. 2, work items) into a pinned device-mapped plan
buffer and one ``ssa_append_attention`` launch (kv_append and the mixed
attention of all requests in one kernel; the same results, bit for bit, as
``ssa_kv_append`` followed by ``ssa_mixed_attention``).  The default
workload is the largest configuration that fits one GPU, the Llama-3-70B-shaped
layer (64 q / 8 kv heads, D = 128, page 16; one 1024-token chunk on a
32768-token prefix plus 32 decodes with contexts uniform in [8192, 32768]),
synthetic and seeded; inputs are resident in HBM before the timed region
starts.

Printed on stdout, as the last line: one JSON object with the metric (µs per
iteration of back-to-back steps), the fused launch's roofline (live timing from
events the kernel stamps itself; bound by whichever floor is larger, the chunk
flops at the bf16 MFMA peak or the algorithmic bytes at the HBM peak, with the
overlap floor and each segment's own fraction beside it), the same launch with
a cold cache, the latency-vs-chunk-size curve (this batch with its chunk cut to
smaller sizes, and the 8B-shaped sweep configuration at three prefixes), the
Llama-3-8B-shaped line for context, and the CPU oracle timed on this host on a
bounded sample (a reported baseline, not the target).

Other modes (all single GPU):
  --sweep OUT        latency-vs-chunk-size table of every workload (JSON lines)
  --copy-probe       plain 1 GiB device copies (the scale of the traffic counters)
  --only-attention   time the attention launch alone (for counter runs; with
                     --fused, the fused launch); --workload, --scene pick the batch
  --pmc-md OUT --pmc-md-dir DIR --pmc-kernel K --pmc-cmd CMD
                     markdown summary of the rocprofv3 counter passes (PMC_PASSES),
                     kernel trace and copy-probe scale collected under DIR
  --traffic-json OUT --traffic-json-inputs F W CF CW
                     HBM traffic summary from rocprofv3 FETCH_SIZE / WRITE_SIZE CSVs
  --sweep-md JSONL   markdown tables of a --sweep file
  --predictor OUT    batch latency predictor (Sec. 3.2, Eq. 5): time the fused
                     launch on random batches of the three scenes, fit the
                     library's predictor on 70% of them, report MAE / RMSE / R^2
                     on the other 30% (as the paper's Tab. 5)
  --chunker OUT      SlidingChunker (Sec. 3.4, Alg. 1) on that predictor: each
                     decision's batch runs on the GPU; reports the measured
                     latency against the prediction and T_cur, and the window
                     cost against the best budget
  --layer OUT        a Llama-3-8B decoder layer on the library's kernels (RMSNorm,
                     projections on the matrix cores, RoPE + kv_append, mixed
                     attention, SwiGLU MLP) vs chunk size, each step timed, the
                     projections also through hipBLASLt for comparison (what the
                     linear layers, Tab. 1's x6 / x7 terms, add to an iteration)
  --layer-predictor OUT
                     Eq. 5 fitted on measured whole-layer times (random batches of
                     the three scenes), with all seven Tab. 1 features and without
                     the linear layers' terms x6, x7
  --peaks OUT        achievable peaks of this GPU (HBM read and copy, bf16 MFMA)
                     from the library's probe kernels, next to the published ones
  --constructor OUT  priority sorter + BatchConstructor (Sec. 3.3, 3.5, Alg. 2):
                     where it reconstructs the batch, the full-budget batch and
                     the constructed one both run on the GPU; reports how many
                     requests meet their TTFT slack in each
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import statistics
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "mixed prefill+decode attention µs/iter vs chunk size; % HBM / MFMA roofline"
HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0
TIME_EVERY = 4  # timed steps whose kernel stamps its start and end
# the sources the fused launch is compiled from (its traffic counters are valid
# only for these exact files)
KERNEL_SRC = [os.path.join(ROOT, "paper_2606_05933_amd", "csrc", f)
              for f in ("ssa_kernels.hip", "ssa_device.h", "ssa_plan_format.h")]
def traffic_file(workload):
    return os.path.join(ROOT, "profiles", f"traffic_append_attention_{workload}.json")

DESCR = {
    "tiny": "tiny mixed: 8q/8kv/D64, 1 chunk (u=192,c=64) + 4 decodes u in {128,256,384,512}",
    "l8b": "Llama-3-8B-shaped mixed layer: 32q/8kv/D128, 1 chunk (u=2048,c=512) + 64 decodes "
           "u~U[512,4096], page 16",
    "l8b_sweep": "Llama-3-8B-shaped chunk sweep: 32q/8kv/D128, 1 chunk of an 8192-token prompt "
                 "+ 128 decodes u~round(LogN(7.0,0.8)) in [64,8192]",
    "multi": "multi-chunk: 28q/4kv/D128, 4 chunks {64,256,512,1024} at u~U[0,8192] + 256 decodes "
             "u~round(LogN(7.2,1.0)) in [64,16384]",
    "l70b": "Llama-3-70B-shaped layer: 64q/8kv/D128, 1 chunk (u=32768,c=1024) + 32 decodes "
            "u~U[8192,32768]",
    "l70b_tp8": "one GPU's share of the Llama-3-70B-shaped layer under 8-way head parallelism: "
                "8q/1kv/D128, 1 chunk (u=32768,c=1024) + 32 decodes u~U[8192,32768]",
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def sha256_file(paths):
    """SHA-256 of one file, or of several files' bytes in order."""
    h = hashlib.sha256()
    for p in ([paths] if isinstance(paths, str) else paths):
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def kernel_event_samples(fn, n, flush=None):
    """Durations (s) of n launches of fn (a DeviceBatch launch method), from
    events that the kernel stamps with its own start and end."""
    import torch
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(n)]
    for a, b in evs:
        a.record()  # creates the HIP events
        b.record()
    for a, b in evs:
        if flush is not None:
            flush()
        fn(events=(a, b))
    torch.cuda.synchronize()
    return [a.elapsed_time(b) / 1e3 for a, b in evs]


def time_kernel_events(fn, n, flush=None):
    """Average duration (s) of n launches of fn (see kernel_event_samples)."""
    return statistics.mean(kernel_event_samples(fn, n, flush))


def percentiles_us(samples_s):
    """Median, 10th and 90th percentile (us) of durations in seconds (nearest rank)."""
    xs = sorted(x * 1e6 for x in samples_s)
    pick = lambda q: xs[min(len(xs) - 1, max(0, int(round(q * (len(xs) - 1)))))]
    return round(statistics.median(xs), 2), round(pick(0.1), 2), round(pick(0.9), 2)


class Flusher:
    """Reads 1 GiB between launches: evicts the L2s and the 256 MB MALL and leaves
    them holding clean lines (a write would leave dirty lines for the measured
    kernel to write back)."""

    def __init__(self):
        import torch
        self.buf = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
        self.acc = torch.zeros((), dtype=torch.float32, device="cuda")

    def __call__(self):
        import torch
        torch.sum(self.buf, dim=(0,), out=self.acc)


def segment_stats(db, n, flush=None):
    us = time_kernel_events(db.attention, n, flush) * 1e6
    info = db.info
    hbm = info.decode_bytes + info.chunk_bytes
    return {"us": round(us, 2), "scene": info.scene,
            "hbm_GBps": round(hbm / us / 1e3, 1), "hbm_frac": round(hbm / us / 1e3 / HBM_PEAK_GBS, 4),
            "mfma_TFLOPs": round(info.chunk_flops / us / 1e6, 1),
            "mfma_frac": round(info.chunk_flops / us / 1e6 / MFMA_BF16_PEAK_TFLOPS, 4)}


def cpu_model():
    """The host CPU's model name (from /proc/cpuinfo)."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def oracle_sample(b, stride):
    """(rows, heads, work of the sample, work of the whole batch): every decode
    row and every stride-th row of each chunk (its last row included), all q
    heads; work counts the (query, key) pairs the oracle visits."""
    starts = np.concatenate([[0], np.cumsum(b.q_len)]).astype(np.int64)
    rows, work, total = [], 0, 0
    for i in range(b.num_reqs):
        c, u = int(b.q_len[i]), int(b.ctx_len[i])
        total += c * (u + 1) + c * (c - 1) // 2
        pick = range(c) if c <= 1 else sorted(set(range(0, c, stride)) | {c - 1})
        for j in pick:
            rows.append(starts[i] + j)
            work += u + j + 1
    hq = b.shape.hq
    rows = np.repeat(np.array(rows, dtype=np.int64), hq)
    heads = np.tile(np.arange(hq, dtype=np.int32), len(rows) // hq)
    return rows, heads, work, total


def cpu_baseline(b, target_s=15.0, threads=0, repeats=3):
    """The fp64 oracle on this host's cores (threads = 0: all the job has): the
    kv_append scatter into copies of the pools (the copy not timed), then
    attention of a bounded sample of the batch's rows, scaled to the whole
    iteration by the (query, key) pairs the oracle visits.  The stride of the
    sampled chunk rows is chosen from a short calibration run so that the
    sample takes about target_s / repeats seconds; the sample is timed
    `repeats` times and the median taken."""
    from oracle import oracle
    s = b.shape
    kc, vc = b.k_cache.copy(), b.v_cache.copy()
    t0 = time.perf_counter()
    oracle.kv_append_inplace(s.hkv, s.d, s.page, b.q_len, b.ctx_len, b.block_table, b.k_new,
                             b.v_new, kc, vc)
    t_app = time.perf_counter() - t0

    def run(stride):
        rows, heads, work, total = oracle_sample(b, stride)
        t = time.perf_counter()
        _, used = oracle.attention_rows(s.hq, s.hkv, s.d, s.page, s.softmax_scale, b.q_len,
                                        b.ctx_len, b.block_table, b.q, kc, vc, rows, heads,
                                        threads=threads)
        return time.perf_counter() - t, used, work, total, len(rows) // s.hq

    max_c = max(1, int(b.q_len.max())) if b.num_reqs else 1
    stride = max(1, max_c // 4)
    each_s = target_s / max(1, repeats)
    dt, used, work, total, nrows = run(stride)  # calibration
    if work < total and dt < each_s:
        # decode rows are always in the sample; the chunk rows' work scales as
        # 1 / stride: pick the stride whose sample takes about each_s
        rate = work / max(dt, 1e-9)
        dec = sum(int(u) + 1 for c, u in zip(b.q_len, b.ctx_len) if c == 1)
        chunk_all = total - dec
        room = each_s * rate - dec
        stride = max(1, int(np.ceil(chunk_all / room))) if room > 0 else max_c
    times = []
    for _ in range(max(1, repeats)):
        dt, used, work, total, nrows = run(stride)
        times.append(dt)
    dt = statistics.median(times)
    t_iter = t_app + dt * total / work
    return {"value": round(t_iter * 1e6, 1), "unit": "us/iter", "cores": int(used),
            "kind": "oracle", "cpu": cpu_model(),
            "sample": f"{b.name}: kv_append of all {b.num_tokens} new rows, then attention of "
                      f"{nrows} of the {b.num_tokens} rows (every decode row, every "
                      f"{stride}th chunk row and the last), all {s.hq} q heads, fp64, "
                      f"median of {len(times)} runs of {dt:.1f} s; scaled by the (query, key) "
                      f"pairs visited ({work} of {total})",
            "tokens_per_s": round(b.num_tokens / t_iter, 1)}


def chunk_row(b, i, c, u):
    """Batch b with request i's chunk cut to its first c tokens at prefix u
    (rows, pools and block table shared; needs c <= b.q_len[i] and
    u + c <= b.ctx_len[i] + b.q_len[i])."""
    from paper_2606_05933_amd import workload
    starts = np.concatenate([[0], np.cumsum(b.q_len)]).astype(np.int64)
    keep = np.concatenate([np.arange(starts[k], starts[k + 1]) if k != i
                           else np.arange(starts[k], starts[k] + c) for k in range(b.num_reqs)])
    q_len, ctx_len = b.q_len.copy(), b.ctx_len.copy()
    q_len[i], ctx_len[i] = c, u
    return workload.Batch(b.shape, q_len, ctx_len, b.block_table, b.num_pages, b.q[keep],
                          b.k_new[keep], b.v_new[keep], b.k_cache, b.v_cache, name=b.name,
                          seed=b.seed)


def chunk_curve(db, rows, n=10):
    """Fused-launch time (us, average of n warm launches) of each (c, u) row
    derived from db's batch (its one chunk request cut to c tokens at prefix u),
    on db's device pools, with the algorithmic rates.  The curve the latency
    predictor and the SlidingChunker consume (Sec. 3.2, 3.4)."""
    from paper_2606_05933_amd.device import DeviceBatch
    b = db.b
    i = int(np.nonzero(b.q_len > 1)[0][0])
    out = []
    for c, u in rows:
        rb = DeviceBatch(chunk_row(b, i, c, u), pools=(db.k_cache, db.v_cache, db.block_table))
        for _ in range(3):
            rb.step_fused()
        t = time_kernel_events(rb.step_fused, n)
        info = rb.info
        nbytes = info.decode_bytes + info.chunk_bytes + info.append_bytes
        out.append({"chunk": int(c), "prefix": int(u), "fused_us": round(t * 1e6, 2),
                    "tokens_per_s": round(rb.b.num_tokens / t, 1),
                    "hbm_frac": round(nbytes / t / 1e9 / HBM_PEAK_GBS, 4),
                    "mfma_frac": round(info.chunk_flops / t / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4)})
        del rb
    return out


def traffic_bytes(workload):
    """HBM bytes per fused launch from committed rocprofv3 counter runs on this
    workload, if they were taken on the current kernel source."""
    f = traffic_file(workload)
    if not os.path.exists(f):
        return None
    t = json.load(open(f))
    if t.get("kernel_source_sha256") != sha256_file(KERNEL_SRC):
        return None
    return (t["fetch_kib"] / t["copy_fetch_factor"] + t["write_kib"] / t["copy_write_factor"]) * 1024


def chunk_launch_bytes(b, info):
    """Algorithmic bytes of the chunk rows' launch of a two-stream iteration:
    the chunk requests' K/V, q and out rows, and the append of their new rows
    (read from k_new / v_new, written to the pools)."""
    s = b.shape
    chunk_tokens = int(b.q_len[b.q_len > 1].sum())
    return info.chunk_bytes + chunk_tokens * s.hkv * s.d * 2 * 2 * 2


def fused_line(db, steps, warmup, streams=False):
    """Back-to-back steps (host plan into the free slot + the iteration's
    launch: the fused launch, or with streams the two-stream pair): wall time
    per step, the average time of the launch that stamps the events (the fused
    launch, or the chunk rows' launch of the pair) on every TIME_EVERY-th step,
    and host time per step."""
    import torch
    launch = db.step_streams if streams else db.step_fused
    for _ in range(warmup):
        db.replan_host()
        launch()
    torch.cuda.synchronize()
    timed = list(range(0, steps, TIME_EVERY))
    evs = {i: [torch.cuda.Event(enable_timing=True) for _ in range(2)] for i in timed}
    for step_evs in evs.values():
        for e in step_evs:
            e.record()  # creates the HIP events
    host_s = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        tp = time.perf_counter()
        db.replan_host()   # host plan into the other (device-mapped) plan slot
        if i in evs:
            launch(events=(evs[i][0], evs[i][1]))
        else:
            launch()
        host_s.append(time.perf_counter() - tp)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    fused_s = statistics.mean(e[0].elapsed_time(e[1]) for e in evs.values()) / 1e3
    return wall / steps, fused_s, statistics.mean(host_s)


def iteration_samples(db, n, flush=None):
    """Durations (s) of n two-stream iterations (db.step_streams), from events
    recorded on the launch stream around each call (the fork to the join)."""
    import torch
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(n)]
    for a, z in evs:
        a.record()
        z.record()
    torch.cuda.synchronize()
    for a, z in evs:
        if flush is not None:
            flush()
        a.record()
        db.step_streams()
        z.record()
    torch.cuda.synchronize()
    return [a.elapsed_time(z) / 1e3 for a, z in evs]


def main_bench(args):
    import torch
    from paper_2606_05933_amd import ssa, workload
    from paper_2606_05933_amd.device import DeviceBatch

    torch.cuda.set_device(0)
    log(f"[bench] generating {args.workload} seed={args.seed}")
    b = workload.make_workload(args.workload, seed=args.seed)
    # the iteration: ssa_append_attention_streams with the planner's choice
    # (mix_order 5): the chunk rows and the decode rows on two streams where
    # that pays, else one launch
    db = DeviceBatch(b, ssa.make_tuning(mix_order=5))
    info = db.info
    split = db.plan_header_field("streams_beside") >= 0 and info.num_chunk_items > 0
    log(f"[bench] items={info.num_items} (chunk {info.num_chunk_items}, decode "
        f"{info.num_decode_items}) groups={info.num_merge_groups} scene={info.scene} "
        f"two streams={split}")

    # the timed region: K back-to-back steps
    step_s, kern_s, host_s = fused_line(db, args.steps, args.warmup, streams=True)
    assert db.status() == 0, "the iteration's launches reported an error"
    # context, after the timed region: the iteration with a cold cache, and the
    # one-launch iteration (ssa_append_attention, the planner's automatic
    # order) warm, cold and as two launches
    flush = Flusher()
    cold = iteration_samples(db, 10, flush)
    cold_p50, cold_p10, cold_p90 = percentiles_us(cold)
    one = DeviceBatch(b, pools=(db.k_cache, db.v_cache, db.block_table))
    one_step_s, fused_s, _ = fused_line(one, 20, 5)
    cold1_p50, cold1_p10, cold1_p90 = percentiles_us(kernel_event_samples(one.step_fused, 10, flush))
    app_s = time_kernel_events(one.kv_append, 20)
    attn_s = time_kernel_events(one.attention, 20)
    assert one.status() == 0, "the one-launch iteration reported an error"
    del one
    tp = time.perf_counter()
    for _ in range(200):
        db._bound[0][0]()
    plan_s = (time.perf_counter() - tp) / 200
    log(f"[bench] step {step_s * 1e6:.1f} us ({'two streams: chunk launch' if split else 'one launch'} "
        f"{kern_s * 1e6:.1f} us), {cold_p50:.1f} us cold; one launch: step "
        f"{one_step_s * 1e6:.1f} us, launch {fused_s * 1e6:.1f} us warm, {cold1_p50:.1f} us cold "
        f"(as two launches: kv_append {app_s * 1e6:.1f} us, attention {attn_s * 1e6:.1f} us); "
        f"host per step {host_s * 1e6:.1f} us, plan {plan_s * 1e6:.1f} us")

    # each segment alone (Eq. 3's pure scenes), cold cache
    segs = {}
    for label, keep in (("decode", b.q_len == 1), ("chunk", b.q_len > 1)):
        if keep.any() and not keep.all():
            sb = DeviceBatch(workload.sub_batch(b, keep))
            sb.step()
            torch.cuda.synchronize()
            segs[label] = segment_stats(sb, 10, flush)
            del sb
            torch.cuda.empty_cache()
    log("[bench] segments alone (cold): "
        + ", ".join(f"{k} {v['us']} us" for k, v in segs.items()))

    # roofline of the dominant kernel: with two streams the chunk rows' launch
    # (its own bytes: the chunk requests' K/V, q, out and appended rows), else
    # the one fused launch (every K/V byte read once, the append's rows read and
    # written once); bytes at the HBM peak, chunk flops at the bf16 MFMA peak,
    # the larger floor names the bound
    all_bytes = info.decode_bytes + info.chunk_bytes + info.append_bytes
    alg_bytes = chunk_launch_bytes(b, info) if split else all_bytes
    t_hbm = alg_bytes / (HBM_PEAK_GBS * 1e9)
    t_mfma = info.chunk_flops / (MFMA_BF16_PEAK_TFLOPS * 1e12)
    tb = traffic_bytes(args.workload)
    if t_mfma > t_hbm:
        achieved = info.chunk_flops / kern_s / 1e12
        roofline = {"bound": "mfma", "achieved": round(achieved, 1),
                    "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                    "frac": round(achieved / MFMA_BF16_PEAK_TFLOPS, 4)}
    else:
        achieved = alg_bytes / kern_s / 1e9
        roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                    "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4)}
    # the whole iteration against its overlap floor: all its bytes at the HBM
    # peak or its flops at the MFMA peak, whichever is larger
    floor = max(all_bytes / (HBM_PEAK_GBS * 1e9), t_mfma)
    roofline.update({
        "traffic": None if tb is None else round(tb),
        "kernel": ("append_attention (the chunk rows' launch of the two-stream iteration)"
                   if split else "append_attention"),
        "kernel_us": round(kern_s * 1e6, 2),
        "algorithmic_bytes": round(alg_bytes), "algorithmic_flops": round(info.chunk_flops),
        "hbm_GBps": round(alg_bytes / kern_s / 1e9, 1),
        "hbm_frac": round(alg_bytes / kern_s / 1e9 / HBM_PEAK_GBS, 4),
        "iteration_us": round(step_s * 1e6, 2),
        "iteration_mfma_frac": round(info.chunk_flops / step_s / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4),
        "iteration_hbm_GBps": round(all_bytes / step_s / 1e9, 1),
        "overlap_floor_us": round(floor * 1e6, 2),
        "frac_of_overlap_floor": round(floor / step_s, 4),
        "sum_of_floors_us": round((all_bytes / (HBM_PEAK_GBS * 1e9) + t_mfma) * 1e6, 2),
        "chunk_segment_mfma_frac": segs.get("chunk", {}).get("mfma_frac"),
        "decode_segment_hbm_frac": segs.get("decode", {}).get("hbm_frac"),
    })

    # latency vs chunk size (the curve the predictor and the SlidingChunker
    # consume): this batch with its chunk cut to smaller sizes, and the 8B-shaped
    # sweep configuration (one 8192-token prompt at prefixes 0 / 2048 / 6144)
    extra = {}
    if not args.no_curve and (b.q_len > 1).any():
        i0 = int(np.nonzero(b.q_len > 1)[0][0])
        cmax, u0 = int(b.q_len[i0]), int(b.ctx_len[i0])
        cs = sorted({c for c in (128, 256, 512) if c < cmax} | {cmax})
        curve = {args.workload: chunk_curve(db, [(c, u0) for c in cs])}
        del db, flush
        torch.cuda.empty_cache()
        bs = workload.make_workload("l8b_sweep", seed=args.seed, chunk=2048, prefix=6144)
        ds = DeviceBatch(bs)
        curve["l8b_sweep"] = chunk_curve(ds, [(c, u) for u in (0, 2048, 6144)
                                              for c in (128, 256, 512, 1024, 2048)])
        del ds, bs
        torch.cuda.empty_cache()
        extra["latency_vs_chunk"] = {
            "note": "fused launch us (average of 10 warm launches) per (chunk, prefix); the "
                    "batch's other requests unchanged", **curve}
        log("[bench] latency vs chunk: " + ", ".join(
            f"{k} c={r['chunk']} u={r['prefix']}: {r['fused_us']} us"
            for k, v in curve.items() for r in v[:3]) + " ...")
        db = flush = None

    # the Llama-3-8B-shaped line (the previous headline), back-to-back steps
    if args.workload != "l8b" and not args.no_extra_line:
        del db, flush
        torch.cuda.empty_cache()
        b8 = workload.make_workload("l8b", seed=args.seed)
        d8 = DeviceBatch(b8)
        s8, f8, _ = fused_line(d8, 20, 5)
        i8 = d8.info
        by8 = i8.decode_bytes + i8.chunk_bytes + i8.append_bytes
        extra["l8b"] = {"workload": DESCR["l8b"], "us_per_iter": round(s8 * 1e6, 2),
                        "fused_us": round(f8 * 1e6, 2),
                        "hbm_GBps": round(by8 / f8 / 1e9, 1),
                        "hbm_frac": round(by8 / f8 / 1e9 / HBM_PEAK_GBS, 4)}
        log(f"[bench] l8b: step {s8 * 1e6:.1f} us, fused {f8 * 1e6:.1f} us")
        del d8
        torch.cuda.empty_cache()

    res = {
        "metric": METRIC, "value": round(step_s * 1e6, 2), "unit": "us/iter",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(step_s * 1e3, 5), "higher_is_better": False, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) bf16 Q/K/V, seeded random block tables; stands in "
                "for the paper's ShareGPT/arXiv request mixes)",
        "config": {"workload": DESCR[args.workload], "name": args.workload, "seed": args.seed,
                   "num_tokens": b.num_tokens, "num_reqs": b.num_reqs,
                   "chunk_tokens": int(b.q_len[b.q_len > 1].sum()),
                   "decode_reqs": int((b.q_len == 1).sum())},
        "tokens_per_s": round(b.num_tokens / step_s, 1),
        "iteration": {"launch": ("ssa_append_attention_streams: chunk rows and decode rows on "
                                 "two streams" if split else "ssa_append_attention (one launch)"),
                      "stamped_launch_us": round(kern_s * 1e6, 2),
                      "cold_us": {"p50": cold_p50, "p10": cold_p10, "p90": cold_p90}},
        "one_launch": {"us_per_iter": round(one_step_s * 1e6, 2),
                       "fused_us": round(fused_s * 1e6, 2),
                       "fused_cold_us": {"p50": cold1_p50, "p10": cold1_p10, "p90": cold1_p90},
                       "two_launch": {"kv_append_us": round(app_s * 1e6, 2),
                                      "attention_us": round(attn_s * 1e6, 2)}},
        "plan_us": round(plan_s * 1e6, 2),
        "host_us_per_step": round(host_s * 1e6, 2),
        "segments_cold": segs,
        "roofline": roofline,
    }
    res.update(extra)
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on this host")
        res["cpu_baseline"] = cpu_baseline(b)
        # single-thread references on the two small configurations
        one = {}
        for name in ("tiny", "l8b"):
            bs = workload.make_workload(name, seed=args.seed)
            r = cpu_baseline(bs, target_s=3.0, threads=1)
            one[name] = {"us_per_iter": r["value"], "sample": r["sample"]}
        res["cpu_baseline"]["one_thread"] = one
    print(json.dumps(res), flush=True)


def sweep_rows(name):
    """(chunk, prefix) rows of the latency-vs-chunk table of a workload; chunk 0 is
    the pure-decode row (Eq. 3)."""
    if name == "tiny":
        return [(c, 192) for c in (0, 16, 32, 64, 128)]
    if name == "l8b":
        return [(c, 2048) for c in (0, 128, 256, 512, 1024, 2048)]
    if name == "l8b_sweep":
        return [(0, 0)] + [(c, u) for u in (0, 2048, 6144) for c in (128, 256, 512, 1024, 2048)]
    if name == "multi":
        return [(0, None)] + [(c, None) for c in (128, 256, 512, 1024)]
    if name in ("l70b", "l70b_tp8"):
        return [(c, 32768) for c in (0, 128, 256, 512, 1024, 2048)]
    raise KeyError(name)


def main_sweep(args):
    import torch
    from paper_2606_05933_amd import workload
    from paper_2606_05933_amd.device import DeviceBatch
    torch.cuda.set_device(0)
    flush = Flusher()
    names = args.sweep_workloads.split(",") if args.sweep_workloads else list(workload.WORKLOADS)
    done = set()
    if os.path.exists(args.sweep):
        for line in open(args.sweep):
            r = json.loads(line)
            done.add((r["workload"], r["chunk"], r["prefix"]))
    out = open(args.sweep, "a")
    for name in names:
        for chunk, prefix in sweep_rows(name):
            if (name, chunk, prefix) in done:
                continue
            b = workload.make_workload(name, seed=args.seed, chunk=chunk, prefix=prefix)
            db = DeviceBatch(b)
            db.step()
            torch.cuda.synchronize()
            n = args.steps
            app = time_kernel_events(db.kv_append, n, flush) * 1e6
            attn_samples = kernel_event_samples(db.attention, n, flush)
            attn = statistics.mean(attn_samples) * 1e6
            p50, p10, p90 = percentiles_us(attn_samples)
            fused = time_kernel_events(db.step_fused, n, flush) * 1e6
            warm = time_kernel_events(db.attention, n) * 1e6
            tp = time.perf_counter()
            for _ in range(n):
                db.replan_host()
            plan = (time.perf_counter() - tp) / n * 1e6
            segs = {}
            for label, keep in (("decode", b.q_len == 1), ("chunk", b.q_len > 1)):
                if keep.any() and not keep.all():
                    sb = DeviceBatch(workload.sub_batch(b, keep))
                    sb.step()
                    torch.cuda.synchronize()
                    segs[label] = segment_stats(sb, n, flush)
                    del sb
            info = db.info
            step_us = plan + fused
            row = {"workload": name, "chunk": chunk, "prefix": prefix, "seed": args.seed,
                   "scene": info.scene, "tokens": b.num_tokens,
                   "attention_us": round(attn, 2), "attention_p50_us": p50,
                   "attention_p10_us": p10, "attention_p90_us": p90,
                   "attention_warm_us": round(warm, 2),
                   "kv_append_us": round(app, 2), "fused_us": round(fused, 2),
                   "plan_us": round(plan, 2),
                   "step_us": round(step_us, 2),
                   "tokens_per_s": round(b.num_tokens / step_us * 1e6, 1),
                   "hbm_GBps": round((info.decode_bytes + info.chunk_bytes) / attn / 1e3, 1),
                   "mfma_TFLOPs": round(info.chunk_flops / attn / 1e6, 1),
                   "decode_bytes": info.decode_bytes, "chunk_flops": info.chunk_flops,
                   "x": list(info.x), "segments": segs,
                   "items": info.num_items}
            out.write(json.dumps(row) + "\n")
            out.flush()
            log(f"[sweep] {name} c={chunk} u={prefix}: attention {attn:.1f} us "
                f"(warm {warm:.1f}), step {step_us:.1f} us, segs "
                + ", ".join(f"{k} {v['us']} us" for k, v in segs.items()))
            del db
            torch.cuda.empty_cache()


def hbm_read_probe(gib: int = 4, workgroups: int = 16384, reps: int = 8) -> float:
    """Achievable HBM read rate (GB/s) on this GPU: ssa_probe_hbm_read streaming
    `gib` GiB (far beyond the 256 MB MALL), best of `reps` launches, timed with
    events around each."""
    import torch
    from paper_2606_05933_amd import ssa
    src = torch.ones((gib << 30) // 4, dtype=torch.float32, device="cuda")
    out = torch.empty(workgroups, dtype=torch.int32, device="cuda")
    best = float("inf")
    for _ in range(reps + 1):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        nbytes = ssa.probe_hbm_read(src, out, workgroups)
        b.record()
        torch.cuda.synchronize()
        best = min(best, a.elapsed_time(b) / 1e3)
    del src, out
    torch.cuda.empty_cache()
    return nbytes / best / 1e9


def main_peaks(args):
    """Achievable peaks of this GPU for the rooflines: HBM read (the library's
    streaming probe over a 4 GiB buffer, several grid sizes), HBM gather (whole
    1, 4 and 16 KB chunks of the same buffer in random order), HBM copy (torch's
    device copy of 1 GiB, read + write bytes), and bf16 MFMA (the library's
    register-only v_mfma_f32_16x16x32_bf16 loop, several grid sizes)."""
    import torch
    from paper_2606_05933_amd import ssa
    torch.cuda.set_device(0)
    res = {"hbm_read_GBps": {}, "mfma_bf16_TFLOPs": {}}
    for wg in (1024, 4096, 16384, 32768, 65536):
        res["hbm_read_GBps"][wg] = round(hbm_read_probe(4, wg), 1)
    src = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    t = []
    for _ in range(9):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        dst.copy_(src)
        b.record()
        torch.cuda.synchronize()
        t.append(a.elapsed_time(b) / 1e3)
    res["hbm_copy_GBps"] = round(2 * (1 << 30) / min(t[1:]) / 1e9, 1)
    del src, dst
    for wg in (256, 512, 1024, 2048, 4096):
        out = torch.empty(wg, dtype=torch.float32, device="cuda")
        best = float("inf")
        for _ in range(6):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            flops = ssa.probe_mfma_bf16(4096, wg, out)
            b.record()
            torch.cuda.synchronize()
            best = min(best, a.elapsed_time(b) / 1e3)
        res["mfma_bf16_TFLOPs"][wg] = round(flops / best / 1e12, 1)
    # gathers of whole chunks in random order over 4 GiB: the decode reads' pattern
    # (4 KB of one page and kv head per load group); 512 workgroups is the attention
    # kernel's residency (two per CU)
    src = torch.ones(1 << 30, dtype=torch.float32, device="cuda")
    res["hbm_gather_GBps"] = {}
    for chunk in (1024, 4096, 16384):
        n = (4 << 30) // chunk
        idx = torch.randperm(n, device="cuda", dtype=torch.int64).to(torch.int32)
        for wg in (512, 4096, 16384):
            out = torch.empty(wg, dtype=torch.int32, device="cuda")
            best = float("inf")
            for _ in range(5):
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record()
                nbytes = ssa.probe_hbm_gather(src, idx, chunk, out, wg)
                b.record()
                torch.cuda.synchronize()
                best = min(best, a.elapsed_time(b) / 1e3)
            res["hbm_gather_GBps"][f"{chunk}B_x{wg}"] = round(nbytes / best / 1e9, 1)
            if chunk == 4096:  # the same chunks read in the key rows' pattern
                best = float("inf")
                for _ in range(5):
                    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                    a.record()
                    nbytes = ssa.probe_hbm_gather(src, idx, chunk, out, wg, pattern=1)
                    b.record()
                    torch.cuda.synchronize()
                    best = min(best, a.elapsed_time(b) / 1e3)
                res["hbm_gather_GBps"][f"{chunk}B_keyrows_x{wg}"] = round(nbytes / best / 1e9, 1)
        del idx
    del src
    torch.cuda.empty_cache()
    res["hbm_read_best_GBps"] = max(res["hbm_read_GBps"].values())
    res["mfma_bf16_best_TFLOPs"] = max(res["mfma_bf16_TFLOPs"].values())
    res["published"] = {"hbm_GBps": HBM_PEAK_GBS, "mfma_bf16_TFLOPs": MFMA_BF16_PEAK_TFLOPS}
    if args.peaks:
        with open(args.peaks, "w") as f:
            json.dump(res, f)
    print(json.dumps(res), flush=True)


def main_copy_probe(args):
    import torch
    torch.cuda.set_device(0)
    src = torch.ones(1 << 28, dtype=torch.float32, device="cuda")  # 1 GiB
    dst = torch.empty_like(src)
    for _ in range(args.steps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": src.numel() * 4, "launches": args.steps}), flush=True)


def main_only_attention(args):
    import torch
    from paper_2606_05933_amd import workload
    from paper_2606_05933_amd.device import DeviceBatch
    torch.cuda.set_device(0)
    b = workload.make_workload(args.workload, seed=args.seed, chunk=args.chunk, prefix=args.prefix)
    if args.scene == "decode":
        b = workload.sub_batch(b, b.q_len == 1)
    elif args.scene == "prefill":
        b = workload.sub_batch(b, b.q_len > 1)
    from paper_2606_05933_amd import ssa
    db = DeviceBatch(b, ssa.make_tuning(mix_order=5) if args.streams else None)
    info = db.info
    for _ in range(3):  # warm-up launches (the trace statistics include them)
        if args.streams:
            db.step_streams()
        else:
            db.step_fused() if args.fused else db.attention()
    if args.streams:
        # the chunk rows' launch of the two-stream iteration (its own stamps)
        us = time_kernel_events(db.step_streams, args.steps) * 1e6
        assert db.status() == 0, "the two-stream launch reported an error"
        kernel, nbytes = "append_attention_kernel", chunk_launch_bytes(b, info)
    elif args.fused:
        # the fused launch appends the rows itself: the algorithmic bytes add them
        us = time_kernel_events(db.step_fused, args.steps) * 1e6
        assert db.status() == 0, "the fused launch reported an error"
        kernel, nbytes = "append_attention_kernel", info.decode_bytes + info.chunk_bytes + info.append_bytes
    else:
        db.kv_append()
        torch.cuda.synchronize()
        us = time_kernel_events(db.attention, args.steps) * 1e6
        kernel, nbytes = "mixed_attention_kernel", info.decode_bytes + info.chunk_bytes
    print(json.dumps({"workload": args.workload, "scene": args.scene, "kernel": kernel,
                      "kernel_us": round(us, 2), "algorithmic_bytes": nbytes,
                      "chunk_flops": info.chunk_flops, "launches": args.steps}), flush=True)


# Counter passes of a --pmc-md summary: rocprofv3 collects one pass per run
# (per-block counter limits), each into DIR/<pass>/run_counter_collection.csv.
PMC_PASSES = {
    "a": "SQ_VALU_MFMA_BUSY_CYCLES SQ_INSTS_VALU_MFMA_MOPS_BF16 SQ_INSTS_MFMA SQ_BUSY_CU_CYCLES "
         "SQ_INSTS_VALU SQ_ACTIVE_INST_VALU SQ_WAVES GRBM_GUI_ACTIVE",
    "b": "SQ_INSTS_LDS SQ_LDS_BANK_CONFLICT SQ_LDS_IDX_ACTIVE SQ_WAIT_INST_LDS "
         "SQ_INSTS_VALU_TRANS_F32 SQ_WAVE_CYCLES GRBM_GUI_ACTIVE",
    "c": "FETCH_SIZE",
    "d": "WRITE_SIZE",
}
NUM_XCC, NUM_SIMD = 8, 1024  # MI355X: 8 dies, 256 CUs x 4 SIMDs


def _pmc_means(path, kernel):
    """Per-dispatch sums of every counter of the kernel's dispatches, averaged."""
    import collections
    import csv
    per = collections.defaultdict(lambda: collections.defaultdict(float))
    for r in csv.DictReader(open(path)):
        if kernel in r["Kernel_Name"]:
            per[r["Dispatch_Id"]][r["Counter_Name"]] += float(r["Counter_Value"])
    if not per:
        raise SystemExit(f"no dispatches of {kernel} in {path}")
    names = set().union(*[set(d) for d in per.values()])
    return {k: statistics.mean(d[k] for d in per.values()) for k in names}, len(per)


def main_pmc_md(args):
    """Markdown summary of the counter passes of one kernel (see PMC_PASSES),
    its kernel-trace statistics and the copy probe's traffic scale."""
    import csv
    d, kernel = args.pmc_md_dir, args.pmc_kernel
    m, nd = {}, {}
    for p in PMC_PASSES:
        vals, n = _pmc_means(os.path.join(d, p, "run_counter_collection.csv"), kernel)
        m.update(vals)
        nd[p] = n
    stats = [r for r in csv.DictReader(open(os.path.join(d, "t", "run_kernel_stats.csv")))
             if kernel in r["Name"]]
    if not stats:
        raise SystemExit(f"no trace statistics of {kernel}")
    calls = int(stats[0]["Calls"])
    dur_ns = float(stats[0]["AverageNs"])
    # per dispatch, in launch order: the first ones are the warm-up launches
    trace = sorted((r for r in csv.DictReader(open(os.path.join(d, "t", "run_kernel_trace.csv")))
                    if kernel in r["Kernel_Name"]), key=lambda r: int(r["Start_Timestamp"]))
    durs = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) for r in trace]
    warm_ns = statistics.mean(durs[3:]) if len(durs) > 3 else dur_ns
    cf, _ = _pmc_means(os.path.join(d, "e", "run_counter_collection.csv"), "copyBuffer")
    cw, _ = _pmc_means(os.path.join(d, "f", "run_counter_collection.csv"), "copyBuffer")
    copy_kib = float(1 << 20)
    f_fac, w_fac = cf["FETCH_SIZE"] / copy_kib, cw["WRITE_SIZE"] / copy_kib
    run = None
    for line in open(os.path.join(d, "t.log")):
        if line.startswith("{"):
            run = json.loads(line)
    gui = m["GRBM_GUI_ACTIVE"] / NUM_XCC  # cycles of one die while the kernel ran
    clock = gui / dur_ns
    mops = m.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0) * 512
    busy = m["SQ_VALU_MFMA_BUSY_CYCLES"] / (gui * NUM_SIMD)
    fetch = m["FETCH_SIZE"] * 1024 / f_fac
    write = m["WRITE_SIZE"] * 1024 / w_fac
    alg_bytes = run["algorithmic_bytes"] if run else None
    alg_flops = run["chunk_flops"] if run else None
    cmd = args.pmc_cmd
    rows = [
        ("dispatches (trace / counter passes a, b, c, d)", f"{calls} / {nd['a']}, {nd['b']}, {nd['c']}, {nd['d']}"),
        ("kernel duration, trace average (all dispatches / after the 3 warm-up launches)",
         f"{dur_ns / 1e3:.1f} / {warm_ns / 1e3:.1f} us"),
        ("GRBM_GUI_ACTIVE per die", f"{gui:.4g} cycles" if args.pmc_concurrent
         else f"{gui:.4g} cycles -> clock {clock:.3f} GHz"),
        ("MFMA busy: SQ_VALU_MFMA_BUSY_CYCLES / (GUI per die x 1024 SIMDs)", f"{busy:.3f}"),
        ("MFMA flops: 512 x SQ_INSTS_VALU_MFMA_MOPS_BF16", f"{mops:.4g}"
         + (f" (algorithmic {alg_flops:.4g})" if alg_flops else "")),
        ("MFMA rate over the trace duration", f"{mops / dur_ns / 1e3:.1f} TFLOP/s = "
         f"{mops / dur_ns / 1e3 / MFMA_BF16_PEAK_TFLOPS:.3f} of {MFMA_BF16_PEAK_TFLOPS:.0f}"
         + ("" if args.pmc_concurrent else
            f" ({mops / dur_ns / 1e3 / (MFMA_BF16_PEAK_TFLOPS * clock / 2.4):.3f} of the peak at {clock:.2f} GHz)")),
        ("SQ_INSTS_MFMA / SQ_WAVES", f"{m['SQ_INSTS_MFMA']:.4g} / {m['SQ_WAVES']:.0f}"),
        ("SQ_BUSY_CU_CYCLES / (GUI per die x 256 CUs)", f"{m['SQ_BUSY_CU_CYCLES'] / (gui * 256):.3f}"),
        ("VALU instructions, SQ_ACTIVE_INST_VALU (quad-cycles)", f"{m['SQ_INSTS_VALU']:.4g}, {m['SQ_ACTIVE_INST_VALU']:.4g}"),
        ("transcendental f32 instructions", f"{m['SQ_INSTS_VALU_TRANS_F32']:.4g}"),
        ("LDS instructions", f"{m['SQ_INSTS_LDS']:.4g}"),
        ("LDS bank-conflict cycles / LDS active cycles", f"{m['SQ_LDS_BANK_CONFLICT']:.4g} / "
         f"{m['SQ_LDS_IDX_ACTIVE']:.4g} = {m['SQ_LDS_BANK_CONFLICT'] / max(m['SQ_LDS_IDX_ACTIVE'], 1):.3f}"),
        ("bank-conflict cycles per LDS instruction", f"{m['SQ_LDS_BANK_CONFLICT'] / max(m['SQ_INSTS_LDS'], 1):.2f}"),
        ("FETCH_SIZE, WRITE_SIZE (KiB per dispatch)", f"{m['FETCH_SIZE']:.6g}, {m['WRITE_SIZE']:.6g}"),
        ("copy probe scale (counter KiB per KiB copied): fetch, write", f"{f_fac:.4f}, {w_fac:.4f}"),
        ("HBM bytes per dispatch (scaled): fetch + write", f"{fetch / 1e6:.1f} + {write / 1e6:.1f} MB"
         + (f" (algorithmic {alg_bytes / 1e6:.1f} MB, ratio {(fetch + write) / alg_bytes:.3f})" if alg_bytes else "")),
        ("HBM rate over the trace duration", f"{(fetch + write) / dur_ns:.0f} GB/s = "
         f"{(fetch + write) / dur_ns / HBM_PEAK_GBS:.3f} of {HBM_PEAK_GBS:.0f}"),
    ]
    out = [f"# {args.pmc_title}", "",
           f"Kernel `{kernel}`; counters averaged over its dispatches.  Workload: "
           + (DESCR.get(run['workload'], run['workload']) + f", scene {run['scene']}" if run else "?") + ".", "",
           "| quantity | value |", "|---|---|"]
    out += [f"| {k} | {v} |" for k, v in rows]
    if args.pmc_concurrent:
        out += ["", "The kernel trace runs the iteration's two streams side by side, so the durations (and",
                "the rates over them) are the kernel's inside the pair.  The counter runs serialise the",
                "two streams' kernels, so the counts are the kernel's own; no clock is derived, since",
                "the two kinds of run differ in timing."]
    out += ["", "Commands (from the repository root, after `cd /tmp && export TMPDIR=/tmp` and back):", "", "```"]
    for p, cs in PMC_PASSES.items():
        out.append(f"rocprofv3 --pmc {cs} -d DIR/{p} -o run --output-format csv -- {cmd}")
    out.append(f"rocprofv3 --kernel-trace --stats -d DIR/t -o run --output-format csv -- {cmd} > DIR/t.log")
    out.append("rocprofv3 --pmc FETCH_SIZE -d DIR/e -o run --output-format csv -- python3 bench.py --copy-probe --steps 3")
    out.append("rocprofv3 --pmc WRITE_SIZE -d DIR/f -o run --output-format csv -- python3 bench.py --copy-probe --steps 3")
    out.append(f"python3 bench.py --pmc-md OUT.md --pmc-md-dir DIR --pmc-kernel {kernel} "
               f"--pmc-cmd '{cmd}' --pmc-title '{args.pmc_title}'"
               + (" --pmc-concurrent" if args.pmc_concurrent else ""))
    out += ["```", ""]
    text = "\n".join(out)
    with open(args.pmc_md, "w") as f:
        f.write(text)
    print(text)


def _pmc_rows(path, counter):
    import csv
    rows = [r for r in csv.DictReader(open(path)) if r["Counter_Name"] == counter]
    return rows


def main_traffic_json(args):
    """HBM traffic of the fused launch from rocprofv3 --pmc runs: FETCH_SIZE and
    WRITE_SIZE (KiB per dispatch) of append_attention_kernel, each scaled by
    what the same counter reads for a plain 1 GiB device copy."""
    fetch, write, cfetch, cwrite = args.traffic_json_inputs
    def kernel_avg(path, counter, name):
        v = [float(r["Counter_Value"]) for r in _pmc_rows(path, counter) if name in r["Kernel_Name"]]
        if not v:
            raise SystemExit(f"no {counter} rows for {name} in {path}")
        return statistics.mean(v), len(v)
    f_kib, n_f = kernel_avg(fetch, "FETCH_SIZE", "append_attention_kernel")
    w_kib, n_w = kernel_avg(write, "WRITE_SIZE", "append_attention_kernel")
    copy_kib = float(1 << 20)  # the copy probe moves 1 GiB
    cf, _ = kernel_avg(cfetch, "FETCH_SIZE", "copyBuffer")
    cw, _ = kernel_avg(cwrite, "WRITE_SIZE", "copyBuffer")
    out = {"kernel": "append_attention_kernel", "workload": DESCR[args.workload],
           "kernel_source_sha256": sha256_file(KERNEL_SRC),
           "fetch_kib": round(f_kib, 1), "write_kib": round(w_kib, 1), "dispatches": [n_f, n_w],
           "copy_fetch_factor": round(cf / copy_kib, 4), "copy_write_factor": round(cw / copy_kib, 4),
           "commands": [f"rocprofv3 --pmc FETCH_SIZE --output-format csv -- {args.pmc_cmd}",
                        f"rocprofv3 --pmc WRITE_SIZE --output-format csv -- {args.pmc_cmd}",
                        "rocprofv3 --pmc FETCH_SIZE --output-format csv -- python3 bench.py --copy-probe --steps 3",
                        "rocprofv3 --pmc WRITE_SIZE --output-format csv -- python3 bench.py --copy-probe --steps 3"]}
    out["traffic_bytes"] = round((out["fetch_kib"] / out["copy_fetch_factor"]
                                  + out["write_kib"] / out["copy_write_factor"]) * 1024)
    json.dump(out, open(args.traffic_json, "w"), indent=1)
    print(json.dumps(out))


# The paper evaluates its predictor on Qwen2.5-7B (Tab. 5): its attention shape
# at one GPU is 28 q / 4 kv heads, D = 128.
PRED_SHAPE = (28, 4, 128)


def predictor_batch(rng, scene):
    """(q_len, ctx_len) of a random batch of one scene (1 pure decode, 2 pure
    prefill, 3 mixed): 1..256 decodes with u ~ round(LogN(7.2, 1.0)) in
    [16, 16384], 1..4 chunks with c ~ U[16, 2048], u ~ U[0, 8192]."""
    nd = 0 if scene == 2 else int(rng.integers(1, 256, endpoint=True))
    npf = 0 if scene == 1 else int(rng.integers(1, 4, endpoint=True))
    c = [int(rng.integers(16, 2048, endpoint=True)) for _ in range(npf)] + [1] * nd
    u = [int(rng.integers(0, 8192, endpoint=True)) for _ in range(npf)] + [
        int(np.clip(np.rint(rng.lognormal(7.2, 1.0)), 16, 16384)) for _ in range(nd)]
    return c, u


def pred_metrics(y, yhat):
    y, yhat = np.asarray(y, dtype=np.float64), np.asarray(yhat, dtype=np.float64)
    r = y - yhat
    ss_tot = float(np.sum((y - y.mean()) ** 2))
    return {"n": int(len(y)), "mae_us": round(float(np.mean(np.abs(r))), 3),
            "rmse_us": round(float(np.sqrt(np.mean(r * r))), 3),
            "r2": round(1.0 - float(np.sum(r * r)) / ss_tot, 5) if ss_tot > 0 else None}


class BatchTimer:
    """Times the fused launch (ssa_append_attention) of arbitrary batches
    {(c_i, u_i)} of one shape: pools, new rows and queries sized once for the
    largest batch, filled with N(0, 1) bf16; each batch gets a random block
    table, a host plan and 2 + 5 launches (the median of the 5, from events the
    kernel stamps itself)."""

    def __init__(self, shape3, max_pages, max_pages_per_req, max_tokens, max_reqs, plan_bytes,
                 ws_bytes, seed):
        import torch
        from paper_2606_05933_amd import ssa
        self.torch, self.ssa = torch, ssa
        hq, hkv, d = shape3
        dev, bf = "cuda", torch.bfloat16
        self.num_pages, self.maxp, self.max_reqs = max_pages, max_pages_per_req, max_reqs
        self.shape = ssa.make_shape(hq, hkv, d, max_pages, max_pages_per_req, d ** -0.5)
        self.kc = torch.empty(max_pages * hkv * 16 * d, dtype=bf, device=dev).normal_()
        self.vc = torch.empty_like(self.kc).normal_()
        self.q = torch.empty(max_tokens * hq * d, dtype=bf, device=dev).normal_()
        self.kn = torch.empty(max_tokens * hkv * d, dtype=bf, device=dev).normal_()
        self.vn = torch.empty_like(self.kn).normal_()
        self.out = torch.empty_like(self.q)
        self.bt = torch.zeros(max_reqs * max_pages_per_req, dtype=torch.int32, device=dev)
        self.ws = torch.zeros(max(ws_bytes, 256), dtype=torch.uint8, device=dev)
        self.plan = torch.zeros(max(plan_bytes, 128), dtype=torch.uint8).pin_memory()
        self.evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                    for _ in range(5)]
        for a, b in self.evs:
            a.record()
            b.record()
        self.rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 12])))

    def time(self, cs, us):
        """(kernel us, plan info) of the batch."""
        torch, ssa = self.torch, self.ssa
        table = np.zeros((self.max_reqs, self.maxp), dtype=np.int32)
        pages = self.rng.permutation(self.num_pages)
        off = 0
        for i, (c, u) in enumerate(zip(cs, us)):
            npg = (u + c + 15) // 16
            table[i, :npg] = pages[off: off + npg]
            off += npg
        torch.cuda.synchronize()
        self.bt.copy_(torch.from_numpy(table.reshape(-1)))
        _, info = ssa.ssa_plan(self.shape, cs, us, out=self.plan)
        call = ssa.bind_append_attention(self.shape, self.plan, self.plan, self.q, self.kn,
                                         self.vn, self.kc, self.vc, self.bt, self.out, self.ws)
        call()
        call()
        for a, b in self.evs:
            call(a, b)
        torch.cuda.synchronize()
        return statistics.median(a.elapsed_time(b) for a, b in self.evs) * 1e3, info


def timer_for(batches, seed):
    """A BatchTimer sized for every (c list, u list) in ``batches``."""
    from paper_2606_05933_amd import ssa
    hq, hkv, d = PRED_SHAPE
    need = [[(u + c + 15) // 16 for c, u in zip(cs, us)] for cs, us in batches]
    num_pages = max(sum(nd) for nd in need) + 64
    maxp = max(max(nd) for nd in need)
    shape = ssa.make_shape(hq, hkv, d, num_pages, maxp, d ** -0.5)
    plan_bytes = ws_bytes = 0
    for cs, us in batches:
        pb, wb = ssa.ssa_plan_size(shape, cs, us)
        plan_bytes, ws_bytes = max(plan_bytes, pb), max(ws_bytes, wb)
    return BatchTimer(PRED_SHAPE, num_pages, maxp, max(sum(cs) for cs, _ in batches),
                      max(len(cs) for cs, _ in batches), plan_bytes, ws_bytes, seed)


def fit_predictor(rows, idx, min_scene):
    from paper_2606_05933_amd import ssa
    p = ssa.Predictor(min_scene_samples=min_scene)
    for i in idx:
        p.add(rows[i]["x"], rows[i]["scene"], rows[i]["us"])
    return p.fit()


def time_batches(timer, batches, tag):
    rows = []
    for k, (scene, cs, us) in enumerate(batches):
        t_us, info = timer.time(cs, us)
        rows.append({"scene": int(info.scene), "x": [float(v) for v in info.x],
                     "us": round(t_us, 3), "reqs": len(cs), "tokens": int(sum(cs))})
        if k % 100 == 99:
            log(f"[{tag}] {k + 1} batches timed")
    return rows


def main_predictor(args):
    import torch
    torch.cuda.set_device(0)
    hq, hkv, d = PRED_SHAPE
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([args.seed, 11])))
    batches = [(1 + k % 3,) + predictor_batch(rng, 1 + k % 3)
               for k in range(args.predictor_samples)]
    timer = timer_for([(cs, us) for _, cs, us in batches], args.seed)
    log(f"[predictor] {len(batches)} batches, pools of {timer.num_pages} pages")
    rows = time_batches(timer, batches, "predictor")
    order = np.random.Generator(np.random.PCG64(args.seed)).permutation(len(rows))
    n_train = int(round(0.7 * len(rows)))
    train, test = order[:n_train], order[n_train:]
    res = {"shape": {"hq": hq, "hkv": hkv, "d": d}, "latency": "ssa_append_attention kernel, us",
           "samples": len(rows), "train": int(len(train)), "test": int(len(test)),
           "min_scene_samples": args.predictor_min_scene, "models": {}}
    for label, min_scene in (("scene experts + global", args.predictor_min_scene),
                             ("global only", 1 << 30)):
        p = fit_predictor(rows, train, min_scene)
        entry = {}
        for split, idx in (("train", train), ("test", test)):
            for sc, name in ((0, "all"), (1, "pure decode"), (2, "pure prefill"), (3, "mixed")):
                sel = [i for i in idx if sc == 0 or rows[i]["scene"] == sc]
                y = [rows[i]["us"] for i in sel]
                yh = [p.predict(rows[i]["x"], rows[i]["scene"]) for i in sel]
                entry[f"{split}/{name}"] = pred_metrics(y, yh)
        entry["coef"] = {m: (None if p.coefficients(m) is None else
                             [float(v) for v in p.coefficients(m)]) for m in range(4)}
        res["models"][label] = entry
    if args.predictor:
        with open(args.predictor, "w") as f:
            json.dump({"summary": res, "rows": rows}, f)
    print(json.dumps(res), flush=True)


class LayerTimer:
    """Times ssa_layer_forward (one Llama-3-8B decoder layer, random weights) on
    arbitrary batches {(c_i, u_i)}: buffers sized once for the largest batch,
    each batch gets a random block table and a host plan; the median of 5
    calls, from events recorded around each call."""

    def __init__(self, batches, seed):
        import torch
        from paper_2606_05933_amd import ssa, workload
        self.torch, self.ssa = torch, ssa
        L = LAYER_DIMS
        hq, hkv, d = L["hq"], L["hkv"], L["d"]
        need = [[(u + c + 15) // 16 for c, u in zip(cs, us)] for cs, us in batches]
        self.num_pages = max(sum(nd) for nd in need) + 64
        self.maxp = max(max(nd) for nd in need)
        self.max_reqs = max(len(cs) for cs, _ in batches)
        max_tokens = max(sum(cs) for cs, _ in batches)
        max_pos = max(u + c for cs, us in batches for c, u in zip(cs, us)) + 1
        self.shape = ssa.make_shape(hq, hkv, d, self.num_pages, self.maxp, d ** -0.5)
        host = workload.layer_weights(seed, L["hidden"], L["inter"], hq, hkv, d)
        self.lw = ssa.LayerWeights(host, hq, hkv, d, max_position=max_pos)
        plan_bytes, ws_bytes = 0, 0
        for cs, us in batches:
            pb, _ = ssa.ssa_plan_size(self.shape, cs, us)
            plan_bytes = max(plan_bytes, pb)
        self.plan = torch.zeros(max(plan_bytes, 128), dtype=torch.uint8).pin_memory()
        for cs, us in batches:
            ssa.ssa_plan(self.shape, cs, us, out=self.plan)
            ws_bytes = max(ws_bytes, ssa.layer_workspace_size(self.shape, self.plan, self.lw))
        dev, bf = "cuda", torch.bfloat16
        self.kc = torch.empty(self.num_pages * hkv * 16 * d, dtype=bf, device=dev).normal_()
        self.vc = torch.empty_like(self.kc).normal_()
        self.x = torch.empty((max_tokens, L["hidden"]), dtype=bf, device=dev).normal_()
        self.out = torch.empty_like(self.x)
        self.bt = torch.zeros(self.max_reqs * self.maxp, dtype=torch.int32, device=dev)
        self.ws = torch.zeros(max(ws_bytes, 256), dtype=torch.uint8, device=dev)
        self.rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 14])))

    def time(self, cs, us):
        """(layer us, plan info) of the batch."""
        torch, ssa = self.torch, self.ssa
        table = np.zeros((self.max_reqs, self.maxp), dtype=np.int32)
        pages = self.rng.permutation(self.num_pages)
        off = 0
        for i, (c, u) in enumerate(zip(cs, us)):
            npg = (u + c + 15) // 16
            table[i, :npg] = pages[off: off + npg]
            off += npg
        torch.cuda.synchronize()
        self.bt.copy_(torch.from_numpy(table.reshape(-1)))
        _, info = ssa.ssa_plan(self.shape, cs, us, out=self.plan)
        t = sum(cs)

        def call():
            ssa.layer_forward(self.shape, self.plan, self.plan, self.lw, self.x[:t], self.out[:t],
                              self.kc, self.vc, self.bt, self.ws)
        (med,) = time_calls([call], 5)
        return med, info


def main_layer_predictor(args):
    """Eq. 5 (per scene, Tab. 1 features) fitted on measured whole-layer times:
    with all seven features, and with the linear layers' terms x6 = sum c and
    x7 = max c removed."""
    import torch
    torch.cuda.set_device(0)
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([args.seed, 15])))
    batches = [(1 + k % 3,) + predictor_batch(rng, 1 + k % 3)
               for k in range(args.predictor_samples)]
    timer = LayerTimer([(cs, us) for _, cs, us in batches], args.seed)
    log(f"[layer-predictor] {len(batches)} batches, pools of {timer.num_pages} pages")
    rows = time_batches(timer, batches, "layer-predictor")
    order = np.random.Generator(np.random.PCG64(args.seed)).permutation(len(rows))
    n_train = int(round(0.7 * len(rows)))
    train, test = order[:n_train], order[n_train:]
    res = {"model": "Llama-3-8B decoder layer (ssa_layer_forward), bf16, random weights",
           "latency": "one layer, us", "samples": len(rows), "train": int(len(train)),
           "test": int(len(test)), "models": {}}
    for label, drop in (("all seven features", ()), ("without x6, x7", (5, 6))):
        rows_d = [dict(r, x=[0.0 if j in drop else v for j, v in enumerate(r["x"])])
                  for r in rows]
        p = fit_predictor(rows_d, train, args.predictor_min_scene)
        entry = {}
        for split, idx in (("train", train), ("test", test)):
            for sc, name in ((0, "all"), (1, "pure decode"), (2, "pure prefill"), (3, "mixed")):
                sel = [i for i in idx if sc == 0 or rows_d[i]["scene"] == sc]
                y = [rows_d[i]["us"] for i in sel]
                yh = [p.predict(rows_d[i]["x"], rows_d[i]["scene"]) for i in sel]
                entry[f"{split}/{name}"] = pred_metrics(y, yh)
        res["models"][label] = entry
    if args.layer_predictor:
        with open(args.layer_predictor, "w") as f:
            json.dump({"summary": res, "rows": rows}, f)
    print(json.dumps(res), flush=True)


# A whole decoder layer takes about 3-5x the attention launch of the same batch
# (profiles/layer_llama3_8b_vs_chunk.md): the latency bounds of the scheduler
# states scale by this when each batch runs as a layer (--timer layer).
LAYER_TIME_SCALE = 4.0


def chunker_state(rng, scale=1.0):
    """A scheduler state: 0..256 decodes (u ~ round(LogN(7.2, 1.0)) in
    [16, 16384]), 1..6 waiting prefills in priority order (cached ~ U[0, 8192],
    remaining ~ U[64, 4096]), the server budget B = |D| + 4096 and the window's
    two latency bounds T_cur, T_next ~ U[60, 400] us (times `scale`)."""
    nd = int(rng.integers(0, 256, endpoint=True))
    dctx = [int(np.clip(np.rint(rng.lognormal(7.2, 1.0)), 16, 16384)) for _ in range(nd)]
    pf = [(int(rng.integers(0, 8192, endpoint=True)), int(rng.integers(64, 4096, endpoint=True)))
          for _ in range(int(rng.integers(1, 6, endpoint=True)))]
    return (dctx, pf, nd + 4096, scale * float(rng.uniform(60, 400)),
            scale * float(rng.uniform(60, 400)))


def timer_of(args, batches):
    """The GPU work each batch runs as: the fused attention launch (default) or a
    whole Llama-3-8B decoder layer (--timer layer)."""
    if args.timer == "layer":
        return LayerTimer(batches, args.seed)
    return timer_for(batches, args.seed)


def main_chunker(args):
    """SlidingChunker (Alg. 1) with a predictor fitted on measured launches:
    each decision's batch is run on the GPU and its measured latency compared
    with the prediction and with T_cur; the chosen window cost is compared with
    the best over every budget (exhaustive, on the host)."""
    import torch
    from paper_2606_05933_amd import ssa
    torch.cuda.set_device(0)
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([args.seed, 13])))
    train = [(1 + k % 3,) + predictor_batch(rng, 1 + k % 3) for k in range(args.predictor_samples)]
    scale = LAYER_TIME_SCALE if args.timer == "layer" else 1.0
    states = [chunker_state(rng, scale) for _ in range(args.chunker_states)]

    def formed(dctx, pf, b, B):
        chunks, _, _ = ssa.form_batch(dctx, pf, b, B)
        cs = [1] * len(dctx) + [c for c in chunks if c > 0]
        us = list(dctx) + [p[0] for p, c in zip(pf, chunks) if c > 0]
        return cs, us

    # the largest batch any decision can form: every decode and every prefill in full
    bound = [formed(d, pf, B, B) for d, pf, B, _, _ in states]
    timer = timer_of(args, [(cs, us) for _, cs, us in train] + [b for b in bound if b[0]])
    rows = time_batches(timer, train, "chunker: predictor samples")
    pred = fit_predictor(rows, range(len(rows)), args.predictor_min_scene)
    out, t_host = [], []
    for k, (dctx, pf, B, t_cur, t_next) in enumerate(states):
        t0 = time.perf_counter()
        b, chunks, t_pred = ssa.sliding_chunker(pred, dctx, pf, B, t_cur, t_next)
        t_host.append(time.perf_counter() - t0)
        b_cur = ssa.time_to_budget(pred, dctx, pf, B, t_cur)
        b_sum = b_cur + ssa.time_to_budget(pred, dctx, pf, B, t_next)

        def pb(x):
            _, feats, sc = ssa.form_batch(dctx, pf, x, B)
            return 0.0 if sc == 0 else pred.predict(feats, sc)
        costs = [pb(x) + pb(b_sum - x) for x in range(len(dctx), min(B, b_cur) + 1)]
        best = min(costs)
        cs, us = formed(dctx, pf, b, B)
        t_meas = timer.time(cs, us)[0] if cs else 0.0
        out.append({"decodes": len(dctx), "prefills": len(pf), "B": B, "t_cur": round(t_cur, 2),
                    "t_next": round(t_next, 2), "b_cur": b_cur, "b_sum": b_sum, "budget": b,
                    "chunks": chunks, "t_pred": round(t_pred, 3), "t_measured": round(t_meas, 3),
                    "window_cost": round(pb(b) + pb(b_sum - b), 3), "window_best": round(best, 3)})
        if k % 50 == 49:
            log(f"[chunker] {k + 1} decisions")
    meas = np.array([o["t_measured"] for o in out])
    prd = np.array([o["t_pred"] for o in out])
    tc = np.array([o["t_cur"] for o in out])
    gap = np.array([(o["window_cost"] - o["window_best"]) / max(o["window_best"], 1e-9)
                    for o in out])
    feasible = np.array([o["b_cur"] > o["decodes"] for o in out])
    res = {"states": len(out), "predictor_samples": len(rows), "timer": args.timer,
           "host_us_per_decision": {"median": round(statistics.median(t_host) * 1e6, 1),
                                    "max": round(max(t_host) * 1e6, 1)},
           "window_cost_gap": {"optimal_fraction": round(float(np.mean(gap <= 1e-12)), 4),
                               "mean": round(float(gap.mean()), 6), "max": round(float(gap.max()), 6)},
           "prediction_error_us": pred_metrics(meas, prd),
           "within_t_cur": {"predicted": round(float(np.mean(prd[feasible] <= tc[feasible])), 4),
                            "measured": round(float(np.mean(meas[feasible] <= tc[feasible])), 4),
                            "states": int(feasible.sum())}}
    if args.chunker:
        with open(args.chunker, "w") as f:
            json.dump({"summary": res, "decisions": out}, f)
    print(json.dumps(res), flush=True)


def constructor_state(rng, scale=1.0):
    """A scheduler state with TTFT pressure: 0..128 decodes (u ~ round(LogN(7.2,
    1.0)) in [16, 16384]), 2..10 prefilling or waiting requests (cached ~
    U[0, 4096], remaining ~ U[32, 1024], TTFT slack ~ U[30, 300] us of this
    path's time (times `scale`), 1 in 10 safeguarded), B = |D| + 4096."""
    nd = int(rng.integers(0, 128, endpoint=True))
    dctx = [int(np.clip(np.rint(rng.lognormal(7.2, 1.0)), 16, 16384)) for _ in range(nd)]
    cands = [(int(rng.integers(0, 4096, endpoint=True)), int(rng.integers(32, 1024, endpoint=True)),
              scale * float(rng.uniform(30, 300)), int(rng.random() < 0.1))
             for _ in range(int(rng.integers(2, 10, endpoint=True)))]
    return dctx, cands, nd + 4096


def main_constructor(args):
    """Multi-Level Priority Sorter + BatchConstructor (Alg. 2) with a predictor
    fitted on measured launches.  Where Alg. 2 reconstructs the batch, both the
    full-budget batch and the constructed one run on the GPU; a candidate meets
    its TTFT if its whole remaining prefill is in the batch and the batch's
    measured time is within its slack."""
    import torch
    from paper_2606_05933_amd import ssa
    torch.cuda.set_device(0)
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([args.seed, 14])))
    train = [(1 + k % 3,) + predictor_batch(rng, 1 + k % 3) for k in range(args.predictor_samples)]
    scale = LAYER_TIME_SCALE if args.timer == "layer" else 1.0
    states = [constructor_state(rng, scale) for _ in range(args.constructor_states)]
    rho, alpha, eps = 20.0, 1.0, 1e-3  # tokens per us of recent throughput; urgency threshold

    def batch_of(dctx, cands, take):
        cs = [1] * len(dctx) + [t for t in take if t > 0]
        us = list(dctx) + [c[0] for c, t in zip(cands, take) if t > 0]
        return cs, us

    bound = [batch_of(d, c, [x[1] for x in c]) for d, c, _ in states]
    timer = timer_of(args, [(cs, us) for _, cs, us in train] + bound)
    rows = time_batches(timer, train, "constructor: predictor samples")
    pred = fit_predictor(rows, range(len(rows)), args.predictor_min_scene)
    outcomes = {0: 0, 1: 0, 2: 0}
    met_full = met_built = risky_total = 0
    t_host, pairs = [], []
    for k, (dctx, cands, B) in enumerate(states):
        t0 = time.perf_counter()
        order = ssa.priority_sort(cands, rho, alpha, eps)
        sc = [cands[i] for i in order]
        outcome, budget, take, t_full = ssa.batch_constructor(pred, dctx, sc, B, eps)
        t_host.append(time.perf_counter() - t0)
        outcomes[outcome] += 1
        if outcome != ssa.CONSTRUCT_BATCH:
            continue
        full_take, _, _ = ssa.form_batch(dctx, [(c[0], c[1]) for c in sc], B, B)
        t_f = timer.time(*batch_of(dctx, sc, full_take))[0]
        t_b = timer.time(*batch_of(dctx, sc, take))[0]
        risky_total += sum(1 for c in sc if c[2] < t_full)
        met_full += sum(1 for c, t in zip(sc, full_take) if t == c[1] and t_f <= c[2])
        met_built += sum(1 for c, t in zip(sc, take) if t == c[1] and t_b <= c[2])
        pairs.append({"t_full_pred": round(t_full, 2), "t_full": round(t_f, 2),
                      "t_built": round(t_b, 2), "budget_full": B, "budget_built": budget,
                      "met_full": sum(1 for c, t in zip(sc, full_take) if t == c[1] and t_f <= c[2]),
                      "met_built": sum(1 for c, t in zip(sc, take) if t == c[1] and t_b <= c[2]),
                      "candidates": len(sc)})
        if k % 50 == 49:
            log(f"[constructor] {k + 1} states")
    res = {"states": len(states), "predictor_samples": len(rows), "timer": args.timer,
           "outcomes": {"no risk": outcomes[0], "no feasible anchor": outcomes[1],
                        "reconstructed": outcomes[2]},
           "host_us_per_decision": {"median": round(statistics.median(t_host) * 1e6, 1),
                                    "max": round(max(t_host) * 1e6, 1)},
           "reconstructed_states": {"candidates_meeting_ttft_full_batch": met_full,
                                    "candidates_meeting_ttft_constructed": met_built,
                                    "risky_candidates": risky_total,
                                    "mean_latency_full_us": round(float(np.mean(
                                        [p["t_full"] for p in pairs])), 2) if pairs else None,
                                    "mean_latency_constructed_us": round(float(np.mean(
                                        [p["t_built"] for p in pairs])), 2) if pairs else None}}
    if args.constructor:
        with open(args.constructor, "w") as f:
            json.dump({"summary": res, "pairs": pairs}, f)
    print(json.dumps(res), flush=True)


LAYER_DIMS = dict(hidden=4096, inter=14336, hq=32, hkv=8, d=128)  # Llama-3-8B
LAYER_CHUNKS = (0, 64, 128, 256, 512, 1024, 2048)


def time_calls(fns, reps):
    """Mean duration (us) of each callable over reps rounds, from event pairs
    recorded around every call on the current stream."""
    import torch
    ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in fns] for _ in range(reps)]
    for f in fns:  # warm up
        f()
    torch.cuda.synchronize()
    for r in range(reps):
        for (a, b), f in zip(ev[r], fns):
            a.record()
            f()
            b.record()
    torch.cuda.synchronize()
    return [statistics.mean(ev[r][i][0].elapsed_time(ev[r][i][1]) for r in range(reps)) * 1e3
            for i in range(len(fns))]


def main_layer(args):
    """One Llama-3-8B decoder layer (ssa_layer_forward: RMSNorm, QKV projection,
    RoPE + kv_append, mixed attention, O projection + residual, RMSNorm, SwiGLU
    MLP + residual; random weights) on the chunk-sweep batches: 128 decodes
    (u ~ round(LogN(7.0, 0.8)) in [64, 8192]) plus one chunk of c tokens of an
    8192-token prompt at prefix 2048.  Reports the layer's latency, each step's
    time, and the same four projections through torch.matmul (hipBLASLt)."""
    import torch
    from paper_2606_05933_amd import ssa, workload
    from paper_2606_05933_amd.device import DeviceBatch
    torch.cuda.set_device(0)
    L = LAYER_DIMS
    host = workload.layer_weights(args.seed, L["hidden"], L["inter"], L["hq"], L["hkv"], L["d"])
    lw = ssa.LayerWeights(host, L["hq"], L["hkv"], L["d"], max_position=8192 + 2048 + 1)
    hid, inter, qd = L["hidden"], L["inter"], L["hq"] * L["d"]
    nqkv = (L["hq"] + 2 * L["hkv"]) * L["d"]
    rows = []
    chunks = LAYER_CHUNKS if args.layer_chunks is None else [int(c) for c in
                                                             args.layer_chunks.split(",")]
    for c in chunks:
        b = workload.make_workload("l8b_sweep", seed=args.seed, chunk=c, prefix=2048)
        db = DeviceBatch(b)
        T = b.num_tokens
        x = torch.from_numpy(workload.normal_bf16((T, hid), args.seed + 7).view(np.int16)).cuda().view(
            torch.bfloat16)
        out = torch.empty_like(x)
        ws = torch.zeros(ssa.layer_workspace_size(db.shape, db.plan_host, lw), dtype=torch.uint8,
                         device="cuda")
        def layer():
            ssa.layer_forward(db.shape, db.plan_host, db.plan_dev, lw, x, out, db.k_cache,
                              db.v_cache, db.block_table, ws)
        (t_layer,) = time_calls([layer], args.steps)
        # the same eight launches captured once in a HIP graph and replayed
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            layer()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            layer()
        (t_graph,) = time_calls([graph.replay], args.steps)
        del graph
        # the steps one by one, on buffers of their own
        bf = dict(dtype=torch.bfloat16, device="cuda")
        xn, qkv, q, a, h = (torch.empty((T, n), **bf) for n in (hid, nqkv, qd, qd, hid))
        act = torch.empty((T, inter), **bf)
        gws = torch.zeros(max(4, max(ssa.linear_workspace_size(T, n, k) for n, k in
                                     ((nqkv, hid), (hid, qd), (2 * inter, hid), (hid, inter)))),
                          dtype=torch.uint8, device="cuda")
        steps = {
            "rms_norm": lambda: ssa.rms_norm(x, lw.attn_norm, xn),
            "qkv": lambda: ssa.linear(xn, lw.w_qkv, qkv, workspace=gws),
            "rope_append": lambda: ssa.rope_append(db.shape, db.plan_host, db.plan_dev, qkv,
                                                   lw.cos_sin, q, db.k_cache, db.v_cache,
                                                   db.block_table),
            "attention": lambda: db.attention(),
            "o_proj": lambda: ssa.linear(a, lw.w_o, h, ssa.EPILOGUE_RESIDUAL, residual=x,
                                         workspace=gws),
            "rms_norm_2": lambda: ssa.rms_norm(h, lw.mlp_norm, xn),
            "gate_up": lambda: ssa.linear(xn, lw.w_gate_up, act, ssa.EPILOGUE_SWIGLU,
                                          workspace=gws),
            "down": lambda: ssa.linear(act, lw.w_down, out, ssa.EPILOGUE_RESIDUAL, residual=h,
                                       workspace=gws),
        }
        t_steps = dict(zip(steps, time_calls(list(steps.values()), args.steps)))
        blas = {"qkv": lambda: torch.matmul(xn, lw.w_qkv.t()),
                "o_proj": lambda: torch.matmul(a, lw.w_o.t()),
                "gate_up": lambda: torch.matmul(xn, lw.w_gate_up.t()),
                "down": lambda: torch.matmul(act, lw.w_down.t())}
        t_blas = dict(zip(blas, time_calls(list(blas.values()), args.steps)))
        lin = sum(t_steps[k] for k in blas)
        flops = 2 * T * (nqkv * hid + hid * qd + 2 * inter * hid + hid * inter)
        row = {"chunk": c, "tokens": T, "decodes": int((b.q_len == 1).sum()),
               "layer_us": round(t_layer, 1), "layer_graph_us": round(t_graph, 1),
               "steps_us": {k: round(v, 1) for k, v in t_steps.items()},
               "linear_us": round(lin, 1), "linear_share": round(lin / sum(t_steps.values()), 3),
               "linear_TFLOPs": round(flops / lin / 1e6, 1),
               "hipblaslt_linear_us": {k: round(v, 1) for k, v in t_blas.items()},
               "hipblaslt_linear_total_us": round(sum(t_blas.values()), 1)}
        rows.append(row)
        log(f"[layer] c={c} T={T} layer={t_layer:.1f}us (graph {t_graph:.1f}us) linear={lin:.1f}us "
            f"(hipBLASLt {sum(t_blas.values()):.1f}us) attention={t_steps['attention']:.1f}us")
        del db, x, out, ws, xn, qkv, q, a, h, act, gws
        torch.cuda.empty_cache()
    tok = np.array([r["tokens"] for r in rows], dtype=np.float64)
    lay = np.array([r["layer_us"] for r in rows])
    slope, icpt = np.polyfit(tok, lay, 1)
    res = {"model": "Llama-3-8B layer (hidden 4096, 32q/8kv/D128, MLP 14336), bf16, random weights",
           "batches": DESCR["l8b_sweep"] + " at prefix 2048", "rows": rows,
           "fit_layer_us": {"per_token": round(float(slope), 4), "intercept": round(float(icpt), 1)}}
    if args.layer:
        with open(args.layer, "w") as f:
            json.dump(res, f)
    print(json.dumps(res), flush=True)


def main_sweep_md(args):
    """Markdown tables of a --sweep JSON-lines file, one per workload."""
    rows = [json.loads(l) for l in open(args.sweep_md) if l.strip()]
    # the row that is the workload's own configuration (multi: chunks scaled by c / 512)
    own = {"tiny": (64, 192), "l8b": (512, 2048), "l70b": (1024, 32768), "multi": (512, None)}
    lines = []
    for name in workload_names_in(rows):
        lines.append(f"### {name}: {DESCR.get(name, name)}\n")
        lines.append("| chunk c | prefix u | scene | tokens | attention us (cold) | "
                     "cold median [p10, p90] | attention us (warm) | "
                     "kv_append us | fused us | plan us | step us | tokens/s | decode-only us | "
                     "chunk-only us | HBM GB/s (% of 8 TB/s) | MFMA TFLOP/s (% of 2.5 PF) | "
                     "floor us: overlap / sum | attention / floor (overlap, sum) |")
        lines.append("|---|---|---|---|---|---|---|---|---|---|---|---|---|---|---|---|---|---|")
        for r in rows:
            if r["workload"] != name:
                continue
            segs = r.get("segments", {})
            dec = segs.get("decode", {}).get("us", "")
            chk = segs.get("chunk", {}).get("us", "")
            mark = " (config)" if own.get(name) == (r["chunk"], r["prefix"]) else ""
            pct = (f"{r['attention_p50_us']} [{r['attention_p10_us']}, {r['attention_p90_us']}]"
                   if "attention_p50_us" in r else "")
            hbm = r["hbm_GBps"]
            tf = r["mfma_TFLOPs"]
            # the mixed launch against its floors at the published peaks: perfect
            # overlap max(bytes / BW, flops / peak), and the sum of the two
            t_mem = r["decode_bytes"] / (HBM_PEAK_GBS * 1e3)
            t_mfma = r["chunk_flops"] / (MFMA_BF16_PEAK_TFLOPS * 1e6)
            f_max, f_sum = max(t_mem, t_mfma), t_mem + t_mfma
            if f_max < 10.0:  # launch- and latency-bound: fractions mean nothing here
                frac = "not meaningful"
            else:
                frac = f"{f_max / r['attention_us']:.0%}, {f_sum / r['attention_us']:.0%}"
            lines.append(
                f"| {r['chunk']}{mark} | "
                f"{r['prefix'] if r['prefix'] is not None else 'drawn'} | {r['scene']} | {r['tokens']} | "
                f"{r['attention_us']} | {pct} | {r['attention_warm_us']} | {r['kv_append_us']} | "
                f"{r.get('fused_us', '')} | {r['plan_us']} | "
                f"{r['step_us']} | {r['tokens_per_s']:.3g} | {dec} | {chk} | "
                f"{hbm} ({hbm / HBM_PEAK_GBS:.0%}) | {tf} ({tf / MFMA_BF16_PEAK_TFLOPS:.0%}) | "
                f"{f_max:.1f} / {f_sum:.1f} | {frac} |")
        lines.append("")
    print("\n".join(lines))


def workload_names_in(rows):
    seen = []
    for r in rows:
        if r["workload"] not in seen:
            seen.append(r["workload"])
    return seen


def main():
    ap = argparse.ArgumentParser(description=__doc__,
                                 formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="l70b")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--chunk", type=int, default=None)
    ap.add_argument("--prefix", type=int, default=None)
    ap.add_argument("--scene", choices=["mixed", "decode", "prefill"], default="mixed")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-curve", action="store_true",
                    help="skip the latency-vs-chunk-size curve of the default line")
    ap.add_argument("--no-extra-line", action="store_true",
                    help="skip the Llama-3-8B-shaped line reported beside the default one")
    ap.add_argument("--sweep", metavar="OUT", default=None)
    ap.add_argument("--sweep-workloads", default=None)
    ap.add_argument("--copy-probe", action="store_true")
    ap.add_argument("--only-attention", action="store_true")
    ap.add_argument("--pmc-concurrent", action="store_true",
                    help="--pmc-md: the traced run has two streams' kernels side by side")
    ap.add_argument("--streams", action="store_true",
                    help="--only-attention: the two-stream iteration (tuning mix_order 5)")
    ap.add_argument("--fused", action="store_true",
                    help="with --only-attention: time the fused launch instead")
    ap.add_argument("--pmc-md", metavar="OUT", default=None,
                    help="markdown summary of rocprofv3 counter passes (see PMC_PASSES)")
    ap.add_argument("--pmc-md-dir", default=None)
    ap.add_argument("--pmc-kernel", default="mixed_attention_kernel")
    ap.add_argument("--pmc-cmd", default="python3 bench.py --only-attention")
    ap.add_argument("--pmc-title", default="Counter summary")
    ap.add_argument("--traffic-json", metavar="OUT", default=None,
                    help="write the HBM traffic summary from four rocprofv3 counter CSVs")
    ap.add_argument("--traffic-json-inputs", nargs=4, metavar=("FETCH", "WRITE", "COPY_FETCH",
                                                               "COPY_WRITE"))
    ap.add_argument("--sweep-md", metavar="JSONL", default=None,
                    help="print the latency-vs-chunk tables of a --sweep file")
    ap.add_argument("--predictor", metavar="OUT", default=None,
                    help="fit and evaluate the batch latency predictor on measured batches")
    ap.add_argument("--predictor-samples", type=int, default=600)
    ap.add_argument("--predictor-min-scene", type=int, default=32)
    ap.add_argument("--chunker", metavar="OUT", default=None,
                    help="SlidingChunker decisions on a measured predictor, run on the GPU")
    ap.add_argument("--chunker-states", type=int, default=200)
    ap.add_argument("--constructor", metavar="OUT", default=None,
                    help="priority sorter + BatchConstructor on a measured predictor, on the GPU")
    ap.add_argument("--constructor-states", type=int, default=300)
    ap.add_argument("--layer", metavar="OUT", default=None,
                    help="a Llama-3-8B decoder layer on the library's kernels vs chunk size")
    ap.add_argument("--timer", choices=["attention", "layer"], default="attention",
                    help="--chunker / --constructor: run each batch as the fused attention "
                         "launch or as a whole Llama-3-8B decoder layer")
    ap.add_argument("--layer-predictor", metavar="OUT", default=None,
                    help="fit Eq. 5 on measured whole-layer times, with and without x6, x7")
    ap.add_argument("--peaks", metavar="OUT", default=None,
                    help="measure the achievable HBM read / copy and bf16 MFMA rates")
    ap.add_argument("--layer-chunks", default=None,
                    help="comma-separated chunk sizes for --layer (default 0,64,...,2048)")
    args = ap.parse_args()
    if args.traffic_json:
        return main_traffic_json(args)
    if args.sweep_md:
        return main_sweep_md(args)
    if args.pmc_md:
        return main_pmc_md(args)
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on one GPU: this attention path has no multi-GPU mode "
              "(head-parallel sharding needs no exchange inside attention); run with --gpus 1.",
              file=sys.stderr)
        sys.exit(2)
    if args.sweep:
        main_sweep(args)
    elif args.copy_probe:
        main_copy_probe(args)
    elif args.only_attention:
        main_only_attention(args)
    elif args.predictor:
        main_predictor(args)
    elif args.chunker:
        main_chunker(args)
    elif args.constructor:
        main_constructor(args)
    elif args.layer:
        main_layer(args)
    elif args.peaks:
        main_peaks(args)
    elif args.layer_predictor:
        main_layer_predictor(args)
    else:
        main_bench(args)


if __name__ == "__main__":
    main()
