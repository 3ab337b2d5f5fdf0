#!/usr/bin/env python3
"""Benchmark: chunked-prefill causal attention on one MI355X.

One step is one layer's attention over a whole synthetic prompt, chunk by chunk
in order (chunk k: plan on the host, then the attention kernel and -- when the
key range is split -- the merge pass), with every input resident in HBM. The
value is the whole job's algorithmic rate: FLOPs of both GEMMs over the visible
(query, key) pairs, 2*Hq*(dqk+dv)*(C*p + C*(C+1)/2) for a chunk of C queries at
prefix p, divided by the wall time of the timed steps.

Besides the contract line it reports, per chunk, the median latency against the
prefix length (the cost curve of sections 4 and 5.1 of the paper) with a
least-squares fit t_k = a + b*k, the residual of the balance identity of Eq. (3)
(t_{k-1} + t_{k+1} - 2 t_k), a roofline entry for the attention kernel (timed
with HIP events on the launch stream) and the fp64 oracle's rate on the host
cores over a bounded sample of the same workload.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload long|mla|gqa|mixed|tiny]

The default workload is the longest single-GPU one: a 524288-token prompt in 32 chunks of
16384 queries, 128 heads of the MLA shape (dqk 192, dv 128), the key range split four ways
with an lse merge; its chunks with a prefix of 64K keys or more (chunks 4..31) are the ones
the 60 %-of-peak target is stated on.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import platform
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "chunked-prefill attention TFLOP/s (% bf16 MFMA peak) + per-chunk latency vs prefix"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0
# per-chunk statistics want >= 20 timed runs; the long and mixed prompts take ~9 s and ~5 s
# per step, so they stop at about a minute of timed work
DEFAULT_STEPS = {"tiny": 50, "gqa": 50, "mla": 20, "long": 6, "mixed": 10}
DEFAULT_WARMUP = {"tiny": 5, "gqa": 5, "mla": 3, "long": 1, "mixed": 1}


def chunk_flops(w, cu, pre):
    """Algorithmic FLOPs of one chunk: both GEMMs over visible pairs."""
    pairs = 0
    for s in range(len(pre)):
        n = int(cu[s + 1] - cu[s])
        p = int(pre[s])
        pairs += n * p + n * (n + 1) // 2
    return 2.0 * w.hq * (w.dqk + w.dv) * pairs, pairs


def chunk_bytes(w, cu, pre):
    """Algorithmic HBM bytes of one chunk: K/V read once, Q read, out and lse written."""
    kv_rows = sum(int(pre[s]) + int(cu[s + 1] - cu[s]) for s in range(len(pre)))
    tok = int(cu[-1])
    return (kv_rows * w.hkv * (w.dqk + w.dv) * 2 + tok * w.hq * w.dqk * 2
            + tok * w.hq * w.dv * 2 + tok * w.hq * 4)


def fit_line(xs, ys):
    n = len(xs)
    if n < 2:
        return None
    mx, my = sum(xs) / n, sum(ys) / n
    sxx = sum((x - mx) ** 2 for x in xs)
    sxy = sum((x - mx) * (y - my) for x, y in zip(xs, ys))
    b = sxy / sxx if sxx else 0.0
    a = my - b * mx
    ss_tot = sum((y - my) ** 2 for y in ys)
    ss_res = sum((y - (a + b * x)) ** 2 for x, y in zip(xs, ys))
    r2 = 1.0 - ss_res / ss_tot if ss_tot else 1.0
    return {"a_ms": a, "b_ms": b, "b_over_a": (b / a) if a else None, "r2": r2}


KERNEL_SRC = os.path.join(ROOT, "paper_2608_26523_amd", "csrc", "vpp_chunk_attn.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "attn_fwd_hbm_bytes.md")


def measured_traffic(workload):
    """HBM bytes per attention launch from the committed FETCH_SIZE/WRITE_SIZE summary,
    scaled by the copy-kernel factors; None unless the summary was taken on the kernel
    source that is here now."""
    import hashlib
    try:
        with open(KERNEL_SRC, "rb") as f:
            sha = hashlib.sha256(f.read()).hexdigest()[:16]
        with open(TRAFFIC_FILE) as f:
            for ln in f:
                parts = ln.split()
                if len(parts) == 4 and parts[0] == "traffic" and parts[1] == workload:
                    return float(parts[3]) if parts[2] == sha else None
    except OSError:
        return None
    return None


def measured_traffic_chunks(workload):
    """HBM bytes of each chunk's attention launch from the same summary (chunk -> bytes);
    None unless it was taken on the kernel source that is here now."""
    import hashlib
    try:
        with open(KERNEL_SRC, "rb") as f:
            sha = hashlib.sha256(f.read()).hexdigest()[:16]
        out = {}
        with open(TRAFFIC_FILE) as f:
            for ln in f:
                parts = ln.split()
                if len(parts) == 5 and parts[0] == "traffic_chunk" and parts[1] == workload:
                    if parts[2] != sha:
                        return None
                    out[int(parts[3])] = float(parts[4])
        return out or None
    except OSError:
        return None


def gemm_reference(dev, n=16384, reps=10):
    """Rate of the platform's own bf16 GEMM (hipBLASLt through torch.matmul) on operands of
    the same kind as the attention inputs (i.i.d. normal) and on zeros. MFMA throughput on
    this part depends on the operand values (power and clock), so this is the ceiling that
    a dense bf16 contraction reaches here on such data; the published peak is not."""
    import torch
    g = torch.Generator(device=dev)
    g.manual_seed(0)
    a = torch.randn((n, n), generator=g, device=dev).to(torch.bfloat16)
    b = torch.randn((n, n), generator=g, device=dev).to(torch.bfloat16)

    def rate(x, y):
        for _ in range(3):
            torch.matmul(x, y)
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            torch.matmul(x, y)
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        return 2.0 * n * n * n / (statistics.median(ts) * 1e-3) / 1e12

    r_randn = rate(a, b)
    z = torch.zeros_like(a)
    r_zeros = rate(z, z)
    del a, b, z
    torch.cuda.empty_cache()
    return {"library": "hipBLASLt via torch.matmul", "shape": "%dx%dx%d bf16" % (n, n, n),
            "randn_tflops": round(r_randn, 1), "zeros_tflops": round(r_zeros, 1)}


def schedule_report(chunk_ms, comm_ms=0.0):
    """Feed a measured per-chunk latency curve (one layer per virtual stage) to the native
    model of the pipeline schedules of sections 2.4 and 5.1-5.3: one request alone under
    each scheme, and two back-to-back copies of it with and without pipelined packing."""
    from paper_2608_26523_amd import schedule as SC
    taus = SC.stage_times_from_curve(chunk_ms)
    out = {"stage_times": "measured per-chunk median latency, one layer per virtual stage",
           "comm_ms": comm_ms}
    for name in ("cpp", "vpp", "vpp_async"):
        r = SC.vpp_sched_simulate([taus], comm_ms, scheme=name)
        out[name] = {"makespan_ms": round(r["makespan"], 4), "bubble_ratio": round(r["bubble_ratio"], 5),
                     "idle_ms": [round(x, 4) for x in r["idle"]]}
    for name in ("vpp_async", "vpp_async_packed"):
        r = SC.vpp_sched_simulate([taus, taus], comm_ms, scheme=name)
        out[name + "_2req"] = {"makespan_ms": round(r["makespan"], 4),
                               "bubble_ratio": round(r["bubble_ratio"], 5),
                               "request_end_ms": [round(x, 4) for x in r["request_end"]]}
    return out


def schedule_sweep(w, q, k, v, sizes, reps=5):
    """Per-chunk latency curves of one prompt of the workload at several chunk sizes
    (the last chunk is shorter when the size does not divide the prompt), each fed to
    the schedule model: the chunk-size sweep of section 6.1."""
    import numpy as np
    import torch
    from paper_2608_26523_amd.attention import ChunkAttention
    S = w.seq_len
    rows = []
    for C in sizes:
        attn = ChunkAttention(w.hq, w.hkv, w.dqk, w.dv, max_chunk_tokens=C, max_kv_len=S,
                              num_splits=w.num_splits)
        out = torch.empty((C, w.hq, w.dv), dtype=torch.bfloat16, device=q.device)
        ms = []
        for c0 in range(0, S, C):
            n = min(C, S - c0)
            cu = np.array([0, n], dtype=np.int32)
            kvs = np.array([0], dtype=np.int64)
            pre = np.array([c0], dtype=np.int64)
            attn.plan(cu, kvs, pre)
            attn.run(q[c0:c0 + n], k, v, out[:n])
            ts = []
            for _ in range(reps):
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record()
                attn.run(q[c0:c0 + n], k, v, out[:n])
                e1.record()
                torch.cuda.synchronize()
                ts.append(e0.elapsed_time(e1))
            ms.append(statistics.median(ts))
        rep = schedule_report(ms)
        rows.append({"chunk": C, "chunks": len(ms), "last_chunk_tokens": S - (len(ms) - 1) * C,
                     "attention_ms": round(sum(ms), 4), "median_ms": [round(x, 4) for x in ms],
                     "schedule": rep})
        del attn, out
    return rows


def build_paged(w, k, v, segs, page, seed=0):
    """Copy the workload's cache into pages of `page` rows, each request's pages in a
    random order, and the per-chunk block tables (one row per segment, in the order of
    the chunk's segments) and slot mappings (where the chunk's own rows go)."""
    import numpy as np
    import torch
    from paper_2608_26523_amd import binding as B
    rng = np.random.default_rng(seed)
    req_rows = {}
    for (_, cu, kvs, pre) in segs:
        for s in range(len(kvs)):
            r = int(kvs[s])
            req_rows[r] = max(req_rows.get(r, 0), int(pre[s]) + int(cu[s + 1] - cu[s]))
    starts = sorted(req_rows)
    npg = {r: (req_rows[r] + page - 1) // page for r in starts}
    total = sum(npg.values())
    perm = rng.permutation(total).astype(np.int32)
    hkv, dqk, dv = k.shape[1], k.shape[2], v.shape[2]
    k_pages = torch.zeros((total, page, hkv, dqk), dtype=k.dtype, device=k.device)
    v_pages = torch.zeros((total, page, hkv, dv), dtype=v.dtype, device=v.device)
    table, pos = {}, 0
    for r in starts:
        ids = perm[pos:pos + npg[r]]
        pos += npg[r]
        table[r] = ids
        rows = req_rows[r]
        full = rows // page
        idx = torch.as_tensor(ids[:full].astype(np.int64), device=k.device)
        if full:
            k_pages.index_copy_(0, idx, k[r:r + full * page].reshape(full, page, hkv, dqk))
            v_pages.index_copy_(0, idx, v[r:r + full * page].reshape(full, page, hkv, dv))
        rem = rows - full * page
        if rem:
            k_pages[int(ids[full]), :rem] = k[r + full * page:r + rows]
            v_pages[int(ids[full]), :rem] = v[r + full * page:r + rows]
    per_chunk = []
    for (_, cu, kvs, pre) in segs:
        width = max(npg[int(x)] for x in kvs)
        bt = np.zeros((len(kvs), width), dtype=np.int32)
        for s in range(len(kvs)):
            ids = table[int(kvs[s])]
            bt[s, :len(ids)] = ids
            bt[s, len(ids):] = ids[0]
        slots = B.vpp_paged_slot_mapping(cu, [0] * len(kvs), pre, bt, page)
        per_chunk.append((torch.as_tensor(bt, device=k.device), torch.as_tensor(slots, device=k.device)))
    return k_pages, v_pages, per_chunk


MFMA_FILE = os.path.join(ROOT, "profiles", "attn_fwd_mfma_clock.md")


def measured_mfma(workload):
    """MFMA pipe utilisation (SQ_VALU_MFMA_BUSY_CYCLES over active cycles of all SIMDs) and the
    shader clock of the attention kernel, from the committed counter summary; None unless it
    was taken on the kernel source that is here now."""
    import hashlib
    try:
        with open(KERNEL_SRC, "rb") as f:
            sha = hashlib.sha256(f.read()).hexdigest()[:16]
        with open(MFMA_FILE) as f:
            for ln in f:
                parts = ln.split()
                if len(parts) == 5 and parts[0] == "mfma" and parts[1] == workload and parts[2] == sha:
                    busy, mhz = float(parts[3]), float(parts[4])
                    # dense bf16 MFMA peak at the clock the kernel actually ran: 256 CUs x
                    # 4096 flop per clock (2.5 PFLOP/s at 2.4 GHz)
                    return {"busy": busy, "clock_mhz": mhz,
                            "busy_vs_peak_clock": round(busy * mhz / 2400.0, 4),
                            "peak_at_clock_tflops": round(256 * 4096 * mhz * 1e6 / 1e12, 1),
                            "source": "rocprofv3 counters, profiles/attn_fwd_mfma_clock.md"}
    except OSError:
        return None
    return None


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def cpu_baseline(w, q, k, v, chunks, budget_s=12.0):
    """Time the fp64 oracle on the host on a bounded sample of the last chunk's items."""
    import numpy as np
    import oracle
    from paper_2608_26523_amd import workloads as W
    oracle.build(force=False)
    kidx = chunks - 1
    t0, cu, kvs, pre = W.chunk_segments(w, kidx)
    tok = int(cu[-1])
    rng = np.random.default_rng(1234)
    # one kv head's group of query heads keeps the host copy small
    g = w.group
    kvh = 0
    hi = max(int(kvs[s] + pre[s] + cu[s + 1] - cu[s]) for s in range(len(pre)))
    qh = q[t0:t0 + tok, kvh * g:(kvh + 1) * g].cpu()
    kh = k[:hi, kvh:kvh + 1].cpu()
    vh = v[:hi, kvh:kvh + 1].cpu()
    threads = oracle.default_threads()
    done_flops, done_items, elapsed = 0.0, 0, 0.0
    batch = max(threads * 2, 16)
    while elapsed < budget_s:
        rows = rng.integers(0, tok, size=batch)
        heads = rng.integers(0, g, size=batch).astype(np.int32)
        seg = np.searchsorted(cu, rows, side="right") - 1
        pos = np.asarray(pre)[seg] + rows - np.asarray(cu)[seg]
        t = time.perf_counter()
        oracle.attention(qh, kh, vh, cu, kvs, pre, rows=rows, heads=heads,
                         scale=w.scale, n_threads=threads)
        elapsed += time.perf_counter() - t
        done_flops += float(np.sum(2.0 * (w.dqk + w.dv) * (pos + 1)))
        done_items += batch
    return {"value": done_flops / elapsed / 1e12, "unit": "TFLOP/s", "cores": threads,
            "kind": "oracle",
            "sample": "%d random (row, head) items of chunk %d (prefix %d) in %.1f s, "
                      "fp64, %s" % (done_items, kidx, int(pre[0]), elapsed, cpu_model())}


def progress(msg):
    """A progress line on stderr (the JSON result is the only line on stdout)."""
    print("bench: " + msg, file=sys.stderr, flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=0)
    ap.add_argument("--warmup", type=int, default=-1)
    ap.add_argument("--workload", default="long")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-gemm-ref", action="store_true",
                    help="skip the library GEMM reference taken after the timed steps")
    ap.add_argument("--chunks", type=int, default=0, help="run only the first N chunks")
    ap.add_argument("--splits", type=int, default=0,
                    help="split count of the key range (-1 automatic, 1 none, 2..16 fixed); "
                         "default: the workload's")
    ap.add_argument("--paged", type=int, default=0,
                    help="page size: run the path over a paged KV cache (pages in random order); "
                         "each chunk first appends its own K/V rows into its pages, then attends")
    ap.add_argument("--mla-split", action="store_true",
                    help="(dqk = 192 workloads) run with the MLA split key layout: per-head k_nope "
                         "[rows, H, 128] and one shared k_rope [rows, 64] (head 0's last 64 dims)")
    ap.add_argument("--schedule-sweep", default="",
                    help="comma-separated chunk sizes: time one prompt of the workload at each "
                         "and print the schedule model's results (one JSON line), nothing else")
    ap.add_argument("--gemm-ref-only", action="store_true",
                    help="only run the library GEMM reference (a known kernel for counter passes)")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="only run a plain device-to-device copy of this many MiB, three "
                         "times (the known-size kernel that scales the HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch
    if args.copy_probe_mib:
        n = args.copy_probe_mib << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": n, "launches": 3}), flush=True)
        return

    if args.gemm_ref_only:
        print(json.dumps(gemm_reference(torch.device("cuda", 0))), flush=True)
        return

    from paper_2608_26523_amd import workloads as W
    from paper_2608_26523_amd.attention import ChunkAttention

    w = W.get(args.workload)
    if args.splits:
        import dataclasses
        w = dataclasses.replace(w, num_splits=args.splits)
    if args.schedule_sweep:
        if w.n_requests != 1:
            print("--schedule-sweep needs a single-request workload", file=sys.stderr)
            sys.exit(2)
        dev = torch.device("cuda", 0)
        torch.cuda.set_device(dev)
        q, k, v = W.make_inputs(w, dev)
        sizes = [int(x) for x in args.schedule_sweep.split(",") if x]
        print(json.dumps({"workload": w.name, "tokens": w.seq_len,
                          "sweep": schedule_sweep(w, q, k, v, sizes)}), flush=True)
        return
    steps = args.steps or DEFAULT_STEPS[w.name]
    warmup = args.warmup if args.warmup >= 0 else DEFAULT_WARMUP[w.name]
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    q, k, v = W.make_inputs(w, dev)
    torch.cuda.synchronize()
    progress("%s inputs resident: q %s, k %s, v %s" % (w.name, tuple(q.shape), tuple(k.shape), tuple(v.shape)))
    S = q.shape[0]
    out = torch.empty((S, w.hq, w.dv), dtype=torch.bfloat16, device=dev)
    lse = torch.empty((w.hq, S), dtype=torch.float32, device=dev)
    nchunks = W.num_chunks(w)
    if args.chunks:
        nchunks = min(nchunks, args.chunks)
    segs = [W.chunk_segments(w, c) for c in range(nchunks)]
    # one plan and one workspace for the whole prompt: every chunk is planned again right
    # before its launch, as a serving loop does (the workspace grows to the largest chunk's)
    attn = ChunkAttention(w.hq, w.hkv, w.dqk, w.dv, max_chunk_tokens=w.chunk, max_kv_len=S,
                          num_splits=w.num_splits)
    splits = [0] * nchunks
    flops = [chunk_flops(w, cu, pre)[0] for (_, cu, _, pre) in segs]
    nbytes = [chunk_bytes(w, cu, pre) for (_, cu, _, pre) in segs]
    stream = torch.cuda.current_stream(dev)
    paged = None
    split_keys = None
    if args.mla_split:
        if w.dqk != 192 or args.paged:
            print("--mla-split needs a dqk = 192 workload and a contiguous cache", file=sys.stderr)
            sys.exit(2)
        split_keys = (k[:, :, :128].contiguous(), k[:, 0, 128:].contiguous())
    if args.paged:
        from paper_2608_26523_amd.attention import kv_append_paged
        paged = build_paged(w, k, v, segs, args.paged)
        append_ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(nchunks)]

    def step(events=None):
        for c, (t0, cu, kvs, pre) in enumerate(segs):
            a = attn
            tok = int(cu[-1])
            if split_keys is not None:
                a.plan(cu, kvs, pre)
                if events is not None:
                    events[c][0].record(stream)
                a.run_mla(q[t0:t0 + tok], split_keys[0], split_keys[1], v, out[t0:t0 + tok],
                          lse[:, t0:t0 + tok], stream=stream)
            elif paged is None:
                a.plan(cu, kvs, pre)
                if events is not None:
                    events[c][0].record(stream)
                a.run(q[t0:t0 + tok], k, v, out[t0:t0 + tok], lse[:, t0:t0 + tok], stream=stream)
            else:
                k_pages, v_pages, per_chunk = paged
                bt, slots = per_chunk[c]
                a.plan(cu, [0] * len(kvs), pre)
                if events is not None:
                    append_ev[c][0].record(stream)
                kv_append_paged(k[t0:t0 + tok], v[t0:t0 + tok], k_pages, v_pages, slots, stream=stream)
                if events is not None:
                    append_ev[c][1].record(stream)
                    events[c][0].record(stream)
                a.run_paged(q[t0:t0 + tok], k_pages, v_pages, bt, out[t0:t0 + tok], lse[:, t0:t0 + tok],
                            stream=stream)
            if events is not None:
                events[c][1].record(stream)

    # the first pass over the chunks is timed on its own: the cold latency (plans built,
    # caches cold); it is one of the warm-up steps when there are any
    cold = None
    if warmup > 0:
        cold_ev = [[torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)]
                   for _ in range(nchunks)]
        step(cold_ev)
        torch.cuda.synchronize()
        cold = [cold_ev[c][0].elapsed_time(cold_ev[c][1]) for c in range(nchunks)]
        progress("cold step done (%.1f ms)" % sum(cold))
    for _ in range(max(0, warmup - 1)):
        step()
    torch.cuda.synchronize()
    progress("%d warm-up step(s) done; timing %d step(s)" % (warmup, steps))
    ev = [[[torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)]
           for _ in range(nchunks)] for _ in range(steps)]
    t_start = time.perf_counter()
    for s in range(steps):
        step(ev[s])
        if steps > 1 and w.name in ("long", "mixed"):
            # the host waits for each step's last event so that the line prints when the
            # step has finished; the next step's first launch then starts from an idle
            # queue (one launch latency, ~0.1 ms of a step of seconds)
            ev[s][-1][1].synchronize()
            progress("timed step %d/%d done" % (s + 1, steps))
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start

    per_chunk = [[ev[s][c][0].elapsed_time(ev[s][c][1]) for s in range(steps)]
                 for c in range(nchunks)]
    med = [statistics.median(x) for x in per_chunk]
    mean = [statistics.fmean(x) for x in per_chunk]
    total_flops = sum(flops)
    ms_per_step = elapsed * 1e3 / steps
    value = total_flops * steps / elapsed / 1e12
    kernel_ms = statistics.fmean(mean)                    # average launch duration
    achieved = (total_flops / nchunks) / (kernel_ms * 1e-3) / 1e12
    for c, (_, cu, kvs, pre) in enumerate(segs):
        splits[c] = attn.plan(cu, kvs if paged is None else [0] * len(kvs), pre).num_splits

    prefix = [int(pre[0]) if len(pre) == 1 else None for (_, _, _, pre) in segs]
    fit = fit_line(list(range(nchunks)), med) if w.n_requests == 1 else None
    eq3 = None
    if w.n_requests == 1 and nchunks >= 3:
        res = [(med[i - 1] + med[i + 1] - 2 * med[i]) / med[i] for i in range(1, nchunks - 1)]
        eq3 = {"mean_rel_residual": statistics.fmean(res), "max_abs_rel_residual": max(abs(r) for r in res)}
    res = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "tokens": S, "chunk": w.chunk, "chunks": nchunks,
                   "requests": w.n_requests, "num_q_heads": w.hq, "num_kv_heads": w.hkv,
                   "head_dim_qk": w.dqk, "head_dim_v": w.dv, "splits": max(splits),
                   "parallelism": "none (1 GPU)"},
        "pct_bf16_peak": round(100.0 * value / PEAK_BF16_TFLOPS, 2),
        "roofline": {"bound": "mfma", "achieved": round(achieved, 3), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": None if (args.paged or args.mla_split) else measured_traffic(w.name),
                     "mfma_util": None if (args.paged or args.mla_split) else measured_mfma(w.name),
                     "kernel": "attn_fwd_kernel", "avg_launch_ms": round(kernel_ms, 4),
                     "flops_per_launch": total_flops / nchunks,
                     "algorithmic_bytes_per_launch": sum(nbytes) / nchunks},
        "kv_cache": ("paged, %d-row pages in random order; each chunk appends its K/V first" % args.paged
                     if args.paged else ("contiguous, MLA split keys (k_nope per head + shared k_rope)"
                                         if args.mla_split else "contiguous")),
        "per_chunk": {"prefix_tokens": prefix, "median_ms": [round(x, 4) for x in med],
                      "min_ms": [round(min(x), 4) for x in per_chunk],
                      "cold_ms": [round(x, 4) for x in cold] if cold else None,
                      "tflops": [round(f / (m * 1e-3) / 1e12, 2) for f, m in zip(flops, med)],
                      # algorithmic bytes over the median time; hbm_gbs: the counter-measured
                      # bytes of the same chunk (committed summary, this kernel source) instead
                      "alg_gbs": [round(b / (m * 1e-3) / 1e9, 1) for b, m in zip(nbytes, med)],
                      "hbm_gbs": None,
                      "splits": splits, "fit": fit, "eq3_residual": eq3},
    }
    tc = None if (args.paged or args.mla_split) else measured_traffic_chunks(w.name)
    if tc is not None and all(c in tc for c in range(nchunks)):
        res["per_chunk"]["hbm_gbs"] = [round(tc[c] / (m * 1e-3) / 1e9, 1) for c, m in enumerate(med)]
    mu = res["roofline"].get("mfma_util")
    if mu:
        mu["frac_at_clock"] = round(achieved / mu["peak_at_clock_tflops"], 4)
    if paged is not None:
        # the last timed step's append kernels: HBM-bound, new K/V rows read and written once
        app_ms = [append_ev[c][0].elapsed_time(append_ev[c][1]) for c in range(nchunks)]
        app_bytes = [2 * int(cu[-1]) * w.hkv * (w.dqk + w.dv) * 2 + 8 * int(cu[-1]) for (_, cu, _, _) in segs]
        gbs = sum(app_bytes) / (sum(app_ms) * 1e-3) / 1e9
        res["kv_append"] = {"kernel": "kv_append_kernel", "bound": "hbm", "avg_launch_ms": round(statistics.fmean(app_ms), 5),
                            "bytes_per_launch": sum(app_bytes) / nchunks, "achieved": round(gbs, 1),
                            "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4)}
    if w.n_requests == 1:
        res["per_chunk"]["schedule_model"] = schedule_report(med)
    if not args.no_gemm_ref:
        ref = gemm_reference(dev)
        ref["attention_frac_of_randn"] = round(achieved / ref["randn_tflops"], 4)
        res["roofline"]["gemm_ref"] = ref
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(w, q, k, v, nchunks)
        # the oracle over the whole timed step, extrapolated from the sampled rate (not run)
        res["cpu_baseline"]["extrapolated_step_s"] = round(total_flops / (res["cpu_baseline"]["value"] * 1e12), 1)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
