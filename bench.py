#!/usr/bin/env python3
"""Replayed anchor tokens/s of SuffixReplay state reconstruction on one MI355X.

A step is one sr_replay_state call over the whole batch: projection GEMM,
conv/gates, conv tail and the chunked scan for every segment and layer of the
workload, inputs already resident in HBM.  Default workload: "varlen16", 16
requests with suffixes of 64*U{8..64} anchor rows, D=2560, H_k=16, H_v=32,
d_k=d_v=128, bf16 (the Qwen3.5-4B linear-layer shape), seeded synthetic data.

Prints ONE JSON line on stdout; progress goes to stderr.

    python bench.py [--gpus 1] [--steps 100] [--warmup 50] [--workload varlen16]
    python bench.py --copy-probe      # plain copy of known size, for HBM counter scaling
    python bench.py --workload sidecar_gather   # anchor sidecar read path (Section 5.2)
    python bench.py --workload sidecar_write    # anchor sidecar write path (Section 5.1)
    python bench.py --workload graph_small      # graph-bucketed replay of a small batch vs eager
    python bench.py --workload group_qwen35_4b  # group replay chaining: 3 layers from one anchor (Section 4.1)
    python bench.py --workload olmo_varlen      # OLMo-Hybrid-7B's d_k=96 / d_v=192 heads (Appendix A)

The two sidecar workloads time the sidecar's own calls instead of the replay
and report anchor rows (x anchored layers) per second, with the HBM roofline
of their dominant kernel.

`roofline.traffic` is the dominant kernel's measured HBM bytes per launch,
read from profiles/traffic_<workload>.json (rocprofv3 FETCH_SIZE / WRITE_SIZE
runs, scaled by what the same counters read for the copy probe); it is null
when that file is missing or was taken from different kernel sources.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))

METRIC = "replayed anchor tokens/sec (state reconstruction) + % MFMA/HBM roofline"

# MI355X published peaks
PEAK_HBM_GBS = 8000.0
PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}


def log(msg):
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


WARMUP_MIN_S = 0.15   # wall time of untimed steps before any timing
BREAKDOWN_STEPS = 20  # untimed steps whose every kernel launch is bracketed by events


def warm_up(step, n):
    """Runs at least n untimed steps, and keeps going (8 at a time, waiting
    for each group) until WARMUP_MIN_S has passed.  From idle the shader
    clock takes ~50-100 ms of this load to settle: timed right after 5
    warmup steps, varlen16 ran 1.43 ms per step, against 1.35-1.37 ms after
    50.  Returns the number of steps run (reported as warmup_run)."""
    import torch
    t0 = time.perf_counter()
    done = 0
    while done < n:
        step()
        done += 1
    torch.cuda.synchronize()
    while time.perf_counter() - t0 < WARMUP_MIN_S:
        for _ in range(8):
            step()
        done += 8
        torch.cuda.synchronize()
    return done


def timed_steps(step, steps, stream):
    """Times `steps` calls of step() between two events on `stream`, with the
    library's HIP events around every launch of the dominant kernel only
    (its live duration is the roofline's); the dominant kernel and the
    others' durations come from BREAKDOWN_STEPS untimed steps just before,
    every launch bracketed.  Events around every kernel inside the timed
    steps would add their own overhead (~20 us per varlen16 step).
    Returns (ms per step, wall ms per step, {kind: (ms, launches)} of the
    breakdown steps with the dominant kind's entry from the timed steps
    scaled to BREAKDOWN_STEPS, dominant kind)."""
    import torch
    import paper_2609_33477_amd as sr
    sr.kernel_timing_kinds(None)
    sr.kernel_timing_enable(True)
    sr.kernel_timing_read()                       # drop anything recorded before
    for _ in range(BREAKDOWN_STEPS):
        step()
    kt = sr.kernel_timing_read()
    dom = max((k for k, (_, n) in kt.items() if n), key=lambda k: kt[k][0])
    sr.kernel_timing_kinds([dom])
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    start.record(stream)
    for _ in range(steps):
        step()
    stop.record(stream)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t_wall) * 1e3 / steps
    tot, n = sr.kernel_timing_read()[dom]
    sr.kernel_timing_enable(False)
    sr.kernel_timing_kinds(None)
    kt[dom] = (tot * BREAKDOWN_STEPS / steps, n * BREAKDOWN_STEPS // steps)
    return start.elapsed_time(stop) / steps, wall, kt, dom


def kernels_timing_note(dom):
    return (f"{dom}: HIP events around each of its launches in the timed steps; the others: "
            f"{BREAKDOWN_STEPS} untimed steps just before, every launch bracketed")


PROJ_LAYERS_PER_LAUNCH = 4   # layers of one call that share a fused-projection launch


def algorithmic_work(wl, with_q=True):
    """Per-launch algorithmic work of each kernel (flops for the MFMA GEMM,
    HBM bytes for the streaming kernels), from the shapes alone."""
    sh = wl.shape
    T = wl.t_total
    D, hk, hv, w = sh.d_model, sh.n_k_heads, sh.n_v_heads, sh.conv_width
    c_kv = hk * sh.d_k + hv * sh.d_v
    N = c_kv + 2 * hv
    es = 4 if sh.anchor_dtype == "f32" else 2             # k/v operand bytes
    wb = {"f32": 4, "bf16": 2, "fp8_e4m3": 1}[sh.weight_dtype]
    tb = 4 if sh.tail_dtype == "f32" else 2
    live = [b for b, s in enumerate(wl.slot_ids) if s >= 0]
    n_layers = len(wl.layers)
    c_q = hk * sh.d_k if with_q else 0
    tail_rows = len(live) * (w - 1)
    # the fused projection covers PROJ_LAYERS_PER_LAUNCH layers per launch:
    # its per-launch work is the average over the call's launches
    proj_layers = n_layers / -(-n_layers // PROJ_LAYERS_PER_LAUNCH)
    return {
        # one launch per layer
        "proj_gemm": ("mfma", 2.0 * T * D * N),
        "conv_gate": ("hbm", T * N * 4 + T * c_kv * es + 2 * T * hv * 4),
        # fused projection + conv epilogue: the contraction is the bound; its
        # HBM traffic is anchors + weights in, k_hat | v | G | beta out.  The
        # q part of the conv tail (a GEMM over the live segments' last w-1
        # rows) runs in the same grid.
        "proj_conv": ("mfma", proj_layers * (2.0 * T * D * N + 2.0 * tail_rows * D * c_q)),
        # fp32 anchors: the tail's own launch
        "tail": ("hbm", c_q * D * wb + tail_rows * ((c_q + c_kv) * tb + D * es)),
        # one launch per call: the varlen tables in, one flag word out, and on
        # the fused path the rows' segment info (16 bytes per row) out
        "validate": ("hbm", (2 * len(wl.seg_lens) + 1) * 4 + 4
                     + (T * 16 if sh.anchor_dtype != "f32" and sh.d_k == sh.d_v else 0)),
        # one launch covers all layers (up to 32)
        "gdn_scan": ("hbm", min(n_layers, 32) * (T * (c_kv * es + hv * 8) + len(live) * hv * sh.d_k * sh.d_v * 4)),
        # the per-head-decay state reads the same operands and writes the same states
        "decay_state": ("hbm", min(n_layers, 32) * (T * (c_kv * es + hv * 8) + len(live) * hv * sh.d_k * sh.d_v * 4)),
    }


# sources each kernel is built from (the traffic record is void once they change)
KERNEL_SOURCES = {
    "proj_conv": ("proj_conv.hip", "tail_q.hpp", "sr_device.hpp", "sr_internal.hpp"),
    "gdn_scan": ("gdn_scan_bf16.hip", "sr_device.hpp", "sr_internal.hpp"),
    "proj_gemm": ("proj_gemm.hip", "sr_device.hpp", "sr_internal.hpp"),
    "decay_state": ("decay_state.hip", "sr_device.hpp", "sr_internal.hpp"),
    "anchor_gather": ("sidecar.hip", "sr_internal.hpp"),
    "anchor_write": ("sidecar.hip", "sr_internal.hpp"),
}


def kernel_source_hash(kernel):
    h = hashlib.sha256()
    for f in KERNEL_SOURCES.get(kernel, ()):
        with open(os.path.join(ROOT, "paper_2609_33477_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(workload, kernel):
    """HBM bytes per launch of `kernel` from the committed counter record, or
    None if there is none for these kernel sources."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    if kernel not in KERNEL_SOURCES or not os.path.exists(path):
        return None
    rec = json.load(open(path)).get("kernels", {}).get(kernel)
    if not rec or rec.get("source_sha256") != kernel_source_hash(kernel):
        return None
    return rec.get("traffic_bytes")


def copy_probe(n_bytes=1 << 30, launches=5):
    """A plain elementwise copy (y = -x over fp32) that reads and writes
    exactly n_bytes each: the reference for scaling FETCH_SIZE / WRITE_SIZE."""
    import torch
    x = torch.ones(n_bytes // 4, dtype=torch.float32, device="cuda")
    y = torch.empty_like(x)
    torch.neg(x, out=y)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(launches):
        torch.neg(x, out=y)
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / launches
    print(json.dumps({"probe": "copy", "read_bytes": n_bytes, "write_bytes": n_bytes, "launches": launches + 1,
                      "avg_ms": round(ms, 4), "GBps": round(2 * n_bytes / (ms * 1e-3) / 1e9, 1)}), flush=True)


def cpu_model():
    """The host CPU's model name (from /proc/cpuinfo), or None."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:  # pragma: no cover
        pass
    return None


def cpu_baseline(wl, budget_s=15.0):
    """The fp64 oracle on a bounded sample of the same workload: whole
    segments, shortest first, until ~budget_s of CPU work.  The projection
    runs on the BLAS threads, the recurrence on the C twin with one host
    thread per value head (up to the cores the process may use)."""
    import numpy as np
    import oracle
    from oracle import crec
    try:
        from threadpoolctl import threadpool_info
        blas = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        blas = 1
    rec_threads = min(crec.threads(), wl.shape.n_v_heads) if crec.available() else 1
    cores = max(blas, rec_threads)
    cu = wl.cu_seqlens
    lay = wl.layers[0]
    rows = 0
    segs = []
    t0 = time.perf_counter()
    for b in np.argsort(wl.seg_lens):          # shortest first keeps the sample bounded
        if time.perf_counter() - t0 > budget_s:
            break
        oracle.replay_segment(wl.shape, lay, lay.anchors[cu[b]:cu[b + 1]])
        rows += wl.seg_lens[b]
        segs.append(int(b))
    el = time.perf_counter() - t0
    rec = (f"recurrence on the C twin over {rec_threads} threads" if crec.available()
           else "recurrence in numpy, single-threaded")
    return {"value": rows / el, "unit": "tokens/s", "cores": int(cores), "kind": "oracle",
            "cpu": cpu_model(),
            "sample": f"{len(segs)} of {len(wl.seg_lens)} segments of layer 0 ({rows} anchor rows, "
                      f"segments {segs}), fp64, {el:.1f} s; projection on {blas} BLAS threads, {rec}"}


SIDECAR_LAYERS = 7      # anchored layers of Qwen3.5-4B (Appendix A: A = G - 1 = 7)
SIDECAR_D = 2560
SIDECAR_PREFILL = (16, 4096)   # write path: a prefill step of 16 requests x 4096 tokens


def bench_sidecar(args):
    """Times the sidecar's gather (the last k anchors of the 16 varlen16
    requests, all 7 anchored layers, into the packed replay batch) or its
    write (compaction + indexed copy of a 64K-token prefill step)."""
    import numpy as np
    import torch
    import workloads as W
    from workloads import sidecar as wsc
    import paper_2609_33477_amd as sr

    def dev(a):
        a = np.ascontiguousarray(a)
        return torch.from_numpy(a.view(np.int16) if a.dtype == np.uint16 else a).cuda()

    A, d, eb = SIDECAR_LAYERS, SIDECAR_D, 2
    row_bytes = d * eb
    stream = torch.cuda.current_stream()
    if args.workload == "sidecar_gather":
        ks = W.make_config("varlen16").seg_lens
        log(f"generating the pool for {len(ks)} requests, {sum(ks)} replay anchors x {A} layers")
        g = wsc.gather_case(0, ks, A, d, eb)
        pool = dev(g.pool)
        sc = sr.make_sidecar(pool, A, wsc.PER_PAGE, d)
        T = int(sum(ks))
        outs = [torch.empty((T, d), dtype=torch.int16, device="cuda") for _ in range(A)]
        cu = torch.empty(len(ks) + 1, dtype=torch.int32, device="cuda")
        tabs = [dev(x) for x in (g.block_table, g.block_cu, g.anchor_first, g.n_anchors)]
        rows = T * A

        def step():
            sr.anchor_gather(sc, *tabs, list(range(A)), outs, cu, stream)

        bytes_of = {"anchor_gather": 2 * rows * row_bytes, "anchor_seqlens": (2 * len(ks) + 1) * 4}
        config = {"workload": args.workload, "requests": len(ks), "anchor_rows": T, "layers": A, "d": d,
                  "elem": "bf16", "per_page": wsc.PER_PAGE, "pool_blocks": g.n_blocks}

        def cpu_leg(budget_s):
            # the oracle's gather over whole requests until the budget is spent
            t0, done, r = time.perf_counter(), 0, 0
            tables = g.block_tables()
            while r < len(ks) and time.perf_counter() - t0 < budget_s:
                from oracle import paged
                paged.anchor_gather(g.pool, A, wsc.PER_PAGE, [tables[r]], [int(g.anchor_first[r])],
                                    [int(ks[r])], list(range(A)))
                done += int(ks[r]) * A
                r += 1
            el = time.perf_counter() - t0
            return {"value": round(done / el, 1), "unit": "anchor rows/s", "cores": 1, "kind": "oracle",
                    "sample": f"oracle.paged.anchor_gather over the first {r} of {len(ks)} requests "
                              f"({done} rows x layers) in {el:.1f} s"}
    elif args.workload == "sidecar_write":
        n_req, L = SIDECAR_PREFILL
        log(f"generating a prefill step of {n_req} x {L} tokens x {A} layers")
        c = wsc.write_case(0, [(0, L)] * n_req, A, d, eb)
        dest_h = sr.anchor_dest_table(c.positions, c.token_req, c.page_table, c.page_cu, wsc.PAGE, wsc.PER_PAGE)
        pool = dev(c.pool)
        sc = sr.make_sidecar(pool, A, wsc.PER_PAGE, d)
        hidden = [dev(h) for h in c.hidden]
        dest = dev(dest_h)
        n = len(dest_h)
        sel = torch.empty(n, dtype=torch.int32, device="cuda")
        n_sel = torch.empty(1, dtype=torch.int32, device="cuda")
        n_rows = int((dest_h >= 0).sum())
        rows = n_rows * A

        def step():
            sr.anchor_compact(dest, sel, n_sel, stream)
            sr.anchor_write(sc, hidden, dest, sel, n_sel, stream)

        bytes_of = {"anchor_compact": n * 4 + n_rows * 4,
                    "anchor_write": 2 * rows * row_bytes + n_rows * 8}
        config = {"workload": args.workload, "requests": n_req, "tokens": n, "anchor_rows": n_rows, "layers": A,
                  "d": d, "elem": "bf16", "per_page": wsc.PER_PAGE}

        def cpu_leg(budget_s):
            from oracle import paged
            t0, done, r = time.perf_counter(), 0, 0
            pool_h = c.pool
            while r < n_req and time.perf_counter() - t0 < budget_s:
                m = c.token_req == r
                sub = paged.compact(np.where(m, dest_h, -1))
                pool_h = paged.anchor_write(pool_h, [h[sub] for h in c.hidden], dest_h[sub], wsc.PER_PAGE)
                done += len(sub) * A
                r += 1
            el = time.perf_counter() - t0
            return {"value": round(done / el, 1), "unit": "anchor rows/s", "cores": 1, "kind": "oracle",
                    "sample": f"oracle.paged compact + anchor_write over the first {r} of {n_req} requests "
                              f"({done} rows x layers) in {el:.1f} s"}
    else:
        raise SystemExit(f"unknown sidecar workload {args.workload}")

    warm_run = warm_up(step, args.warmup)
    ms_per_step, _, kt, dom = timed_steps(step, args.steps, stream)
    kernels = {}
    for k, (tot, cnt) in kt.items():
        if cnt == 0:
            continue
        avg_ms = tot / cnt
        ach = bytes_of[k] / (avg_ms * 1e-3) / 1e9
        kernels[k] = {"avg_ms": round(avg_ms, 5), "launches_per_step": cnt / BREAKDOWN_STEPS,
                      "share": round(tot / max(sum(v[0] for v in kt.values()), 1e-12), 4), "bound": "hbm",
                      "bytes": bytes_of[k], "achieved": round(ach, 2), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                      "frac": round(ach / PEAK_HBM_GBS, 4)}
    dk = kernels[dom]
    roofline = {"bound": "hbm", "achieved": dk["achieved"], "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": dk["frac"], "traffic": measured_traffic(args.workload, dom), "kernel": dom}
    value = rows / (ms_per_step / 1e3)
    log(f"{ms_per_step:.4f} ms/step, {value / 1e6:.2f} M rows/s; {dom} {dk['achieved']:.0f} GB/s")
    cpu = None if args.no_cpu_baseline else cpu_leg(min(args.cpu_budget_s, 15.0))
    out = {"metric": f"anchor rows x layers/sec ({args.workload.replace('_', ' ')})", "value": round(value, 1),
           "unit": "rows/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "warmup_run": warm_run,
           "ms_per_step": round(ms_per_step, 5), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
           "dtype": "bf16", "data": "synthetic", "config": config, "latency_ms": round(ms_per_step, 5),
           "roofline": roofline, "kernels": kernels, "kernels_timing": kernels_timing_note(dom), "cpu_baseline": cpu}
    print(json.dumps(out), flush=True)


GRAPH_SEGMENTS = [128] * 8          # a small batch of hits: 8 requests x 128 replayed anchors
GRAPH_LAYERS = 24                   # every linear-attention layer of Qwen3.5-4B (Appendix A)
GRAPH_GROUPS = 8                    # its 8 groups of 3 linear layers (G = 8 full-attention layers)
GRAPH_BUCKETS = [256, 1024, 4096]   # total-length buckets, up to the paper's T_max = 4096
GRAPH_MIN_WARMUP = 100              # untimed batches per mode before timing (at least)


def bench_graph(args):
    """Replay of a small batch of hits (8 x 128 anchors through all 24
    Qwen3.5-4B linear layers, 8 groups of 3) through the graph-bucketed path
    (one sr_replay_graph per group: graphs captured at creation, one shared
    workspace), with each group's anchors fetched from pinned host memory on
    a copy stream while the previous group replays (Section 5.2).  Reports
    the pipelined fetch + replay wall time per batch against the fetch alone,
    the replay alone (anchors resident) and the eager sr_replay_state call."""
    import torch
    import workloads as W
    from workloads.device import upload
    import paper_2609_33477_amd as sr

    shape = W.config_shape("varlen16")[0]
    per = GRAPH_LAYERS // GRAPH_GROUPS
    wl = W.make_workload("graph_small", shape, GRAPH_SEGMENTS, n_layers=GRAPH_LAYERS, seed=3)
    dev = upload(wl)
    layers = [sr.LayerTensors(**vars(ns)) for ns in dev.layers]
    ws_group = torch.empty(sr.replay_workspace_size(shape, per, GRAPH_BUCKETS[-1]), dtype=torch.uint8,
                           device="cuda")
    groups = [sr.ReplayGraph(shape, layers[g * per:(g + 1) * per], max_segments=len(GRAPH_SEGMENTS),
                             bucket_rows=GRAPH_BUCKETS, workspace=ws_group) for g in range(GRAPH_GROUPS)]
    host = [dev.layers[li].anchors.view(torch.int16).cpu().pin_memory() for li in range(GRAPH_LAYERS)]
    ws_bytes = sr.replay_workspace_size(shape, GRAPH_LAYERS, wl.t_total)
    ws = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device="cuda")
    stream, copy_stream = torch.cuda.current_stream(), torch.cuda.Stream()
    n = len(GRAPH_SEGMENTS)
    ranges = [[(host[g * per + i], i, 0) for i in range(per)] for g in range(GRAPH_GROUPS)]

    def eager():
        sr.replay_state(shape, layers, n, wl.t_total, dev.cu_seqlens, dev.slot_ids, ws, ws_bytes, stream)

    def replay_only():
        for g in groups:
            g.run(n, wl.t_total, dev.cu_seqlens, dev.slot_ids, stream)

    def fetch_only():
        for g, r in zip(groups, ranges):
            g.fetch(r, copy_stream)
        stream.wait_stream(copy_stream)

    def pipelined():
        for g, r in zip(groups, ranges):
            g.fetch(r, copy_stream)
            g.run(n, wl.t_total, dev.cu_seqlens, dev.slot_ids, stream)

    warm_runs = []

    def timed(fn):
        # The first ~60 pipelined batches of a process run ~25% slower: the
        # runtime blocks the host inside the copy submissions until it has
        # warmed up, and the copy stream idles between copies.  Warm every
        # mode past that point.
        warm_runs.append(warm_up(fn, max(args.warmup, GRAPH_MIN_WARMUP)))
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        a.record(stream)
        for _ in range(args.steps):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / args.steps, (time.perf_counter() - t0) * 1e3 / args.steps

    ms_pipe, wall_pipe = timed(pipelined)
    ms_fetch, _ = timed(fetch_only)
    ms_replay, _ = timed(replay_only)
    ms_eager, _ = timed(eager)
    # the kernels' own durations, from the eager path's per-kernel events
    sr.kernel_timing_enable(True)
    sr.kernel_timing_read()
    for _ in range(args.steps):
        eager()
    kt = sr.kernel_timing_read()
    sr.kernel_timing_enable(False)
    work = algorithmic_work(wl, with_q=dev.with_q)
    tot, cnt = kt["proj_conv"]
    avg_ms = tot / cnt
    ach = work["proj_conv"][1] / (avg_ms * 1e-3) / 1e12
    for g in groups:
        g.close()
    fetched = sum(h.numel() * h.element_size() for h in host)
    value = wl.replayed_tokens / (ms_pipe / 1e3)
    log(f"pipelined fetch+replay {ms_pipe:.4f} ms (wall {wall_pipe:.4f}), fetch {ms_fetch:.4f} ms "
        f"({fetched / ms_fetch / 1e6:.1f} GB/s), replay {ms_replay:.4f} ms, sum {ms_fetch + ms_replay:.4f} ms, "
        f"eager replay {ms_eager:.4f} ms")
    out = {"metric": METRIC + " (graph-bucketed small batch, anchors fetched from host)", "value": round(value, 1),
           "unit": "tokens/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "warmup_run": warm_runs[0],
           "ms_per_step": round(ms_pipe, 5), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
           "dtype": "bf16", "data": "synthetic",
           "config": {"workload": "graph_small", "requests": n, "anchors_per_request": GRAPH_SEGMENTS[0],
                      "layers": GRAPH_LAYERS, "groups": GRAPH_GROUPS,
                      "t_total": wl.t_total, "bucket_rows": GRAPH_BUCKETS, "d_model": shape.d_model,
                      "n_k_heads": shape.n_k_heads, "n_v_heads": shape.n_v_heads, "d_k": shape.d_k},
           "latency_ms": round(ms_pipe, 5),
           "pipeline": {"fetch_replay_ms": round(ms_pipe, 5), "fetch_ms": round(ms_fetch, 5),
                        "replay_ms": round(ms_replay, 5), "sum_ms": round(ms_fetch + ms_replay, 5),
                        "eager_replay_ms": round(ms_eager, 5), "fetched_bytes": fetched,
                        "fetch_GBps": round(fetched / ms_fetch / 1e6, 1)},
           "roofline": {"bound": "mfma", "achieved": round(ach, 2), "peak": PEAK_TFLOPS["bf16"], "unit": "TFLOP/s",
                        "frac": round(ach / PEAK_TFLOPS["bf16"], 4), "traffic": None, "kernel": "proj_conv"},
           "cpu_baseline": None}
    print(json.dumps(out), flush=True)


GROUP_SEGMENTS = [512] * 8          # 8 hits at the Qwen3.5-4B replay cap (k_max = 512): T_max = 4096 rows


def group_work(gw):
    """Per-launch algorithmic work of each group-replay kernel (flops for
    the MFMA kernels, HBM bytes for the streaming ones), summed over the
    call's launches of that kernel."""
    sh = gw.shape
    T, D, hk, hv, d, F = gw.t_total, sh.d_model, sh.n_k_heads, sh.n_v_heads, sh.d_k, gw.d_ff
    n = len(gw.blocks)
    live = [b for b, s in enumerate(gw.slot_ids) if s >= 0]
    n_full = (hk + hk + hv + hv) * d + 2 * hv          # q | k | v | z | a | b
    n_last = (hk + hv) * d + 2 * hv                    # k | v | a | b
    C = 64                                             # chunk rows of the output kernel
    # chunk form: four C^2 d-sized products (K K^T, Q K^T, T diag(beta) R,
    # (P o Q K^T) Delta) and three C d^2-sized ones (K M0, Q M0, K^T Delta);
    # the kernel runs them as bf16 hi/lo split products on the bf16 MFMA
    per_row_head = 8 * C * d + 6 * d * d
    tail_rows = len(live) * (sh.conv_width - 1)
    return {
        # the last layer's projection grid also runs the q part of the conv tail
        "proj_conv": ("mfma", 2.0 * T * D * (n_full * (n - 1) + n_last) + 2.0 * tail_rows * D * hk * d),
        "gdn_output": ("mfma", float(per_row_head) * T * hv * (n - 1)),
        "gemm_resid": ("mfma", 2.0 * T * D * (hv * d + F) * (n - 1)),
        "gemm_swiglu": ("mfma", 2.0 * T * D * 2 * F * (n - 1)),
        # input norm of every layer, post-mixer norm of every layer but the last
        "rmsnorm": ("hbm", T * D * ((2 + 2 + 4) + (n - 1) * (4 + 2) + (n - 1) * (4 + 2))),
        "gdn_scan": ("hbm", T * ((hk + hv) * d * 2 + hv * 8) + len(live) * hv * d * d * 4),
        # the table check, with the rows' segment info in the same launch
        "validate": ("hbm", (2 * len(gw.seg_lens) + 1) * 4 + 4 + T * 16),
    }


def bench_group(args):
    """Group replay chaining (Section 4.1): a 3-layer group at Qwen3.5-4B's
    shape rebuilt from its group-entry anchors, for 8 hits of 512 anchors."""
    import torch
    import workloads as W
    from workloads.device import upload_group
    from workloads.group import make_group
    import paper_2609_33477_amd as sr

    shape = W.config_shape("varlen16")[0]
    gw = make_group("group_qwen35_4b", shape, GROUP_SEGMENTS, seed=6)
    dg = upload_group(gw)
    blocks = [sr.BlockTensors(**vars(b)) for b in dg.blocks]
    ws_bytes = sr.group_workspace_size(shape, gw.d_ff, gw.t_total)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()
    n_seg = len(gw.seg_lens)

    def step():
        sr.replay_group(shape, gw.d_ff, gw.norm_eps, blocks, dg.anchors, n_seg, gw.t_total, dg.cu_seqlens,
                        dg.slot_ids, ws, ws_bytes, stream)

    log(f"group: T={gw.t_total} rows x {len(blocks)} layers, d_ff {gw.d_ff}, workspace {ws_bytes / 2**20:.1f} MiB")
    warm_run = warm_up(step, args.warmup)
    ms, _, kt, dom = timed_steps(step, args.steps, stream)
    value = gw.replayed_tokens / (ms / 1e3)
    log(f"{ms:.3f} ms/step, {value / 1e6:.2f} M tokens/s (rows x layers)")
    work = group_work(gw)
    kernels = {}
    for k, (tot, cnt) in kt.items():
        if cnt == 0:
            continue
        bound, amount = work[k]
        step_ms = tot / BREAKDOWN_STEPS                      # all launches of the kind in one step
        if bound == "mfma":
            ach, peak, unit = amount / (step_ms * 1e-3) / 1e12, PEAK_TFLOPS["bf16"], "TFLOP/s"
        else:
            ach, peak, unit = amount / (step_ms * 1e-3) / 1e9, PEAK_HBM_GBS, "GB/s"
        kernels[k] = {"ms_per_step": round(step_ms, 5), "launches_per_step": cnt / BREAKDOWN_STEPS,
                      "share": round(tot / max(sum(v[0] for v in kt.values()), 1e-12), 4),
                      "bound": "mfma" if bound.startswith("mfma") else bound, "achieved": round(ach, 2),
                      "peak": peak, "unit": unit, "frac": round(ach / peak, 4)}
    dk = kernels[dom]
    cpu = None
    if not args.no_cpu_baseline:
        from oracle import block
        log("timing the fp64 oracle on a bounded sample")
        t0 = time.perf_counter()
        cu = gw.cu_seqlens
        rows = 0
        for b in range(n_seg):
            if time.perf_counter() - t0 > args.cpu_budget_s:
                break
            block.replay_group_segment(shape, gw.blocks, gw.anchors[cu[b]:cu[b + 1]], gw.norm_eps)
            rows += gw.seg_lens[b]
        el = time.perf_counter() - t0
        cpu = {"value": rows * len(blocks) / el, "unit": "tokens/s", "kind": "oracle", "cpu": cpu_model(),
               "cores": int(os.cpu_count() or 1),
               "sample": f"{rows} anchor rows of {n_seg} segments through {len(blocks)} layers, fp64, {el:.1f} s"}
    out = {"metric": METRIC + " (group replay chaining)", "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "warmup_run": warm_run, "ms_per_step": round(ms, 4),
           "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
           "config": {"workload": gw.name, "requests": n_seg, "anchors_per_request": GROUP_SEGMENTS[0],
                      "layers": len(blocks), "t_total": gw.t_total, "d_model": shape.d_model,
                      "n_k_heads": shape.n_k_heads, "n_v_heads": shape.n_v_heads, "d_k": shape.d_k,
                      "d_ff": gw.d_ff},
           "latency_ms": round(ms, 4),
           "roofline": {"bound": dk["bound"], "achieved": dk["achieved"], "peak": dk["peak"], "unit": dk["unit"],
                        "frac": dk["frac"], "traffic": None, "kernel": dom},
           "kernels": kernels, "kernels_timing": kernels_timing_note(dom), "cpu_baseline": cpu}
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    # the clock needs ~50 steps (~80 ms of this load) to settle: warm_up
    # runs at least --warmup steps and at least WARMUP_MIN_S of them
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--workload", default="varlen16")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget-s", type=float, default=15.0)
    ap.add_argument("--copy-probe", action="store_true", help="time a plain 1 GiB copy and exit")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one MI355X: the replay path here runs on a single GPU "
              f"(--gpus {args.gpus}, WORLD_SIZE {world} requested). Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    if args.copy_probe:
        copy_probe()
        return
    if args.workload.startswith("sidecar_"):
        bench_sidecar(args)
        return
    if args.workload == "graph_small":
        bench_graph(args)
        return
    if args.workload == "group_qwen35_4b":
        bench_group(args)
        return

    import torch
    import workloads as W
    from workloads.device import upload
    import paper_2609_33477_amd as sr

    log(f"generating workload {args.workload}")
    wl = W.make_config(args.workload)
    dev = upload(wl)
    ws_bytes = sr.replay_workspace_size(wl.shape, len(wl.layers), wl.t_total)
    ws = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device="cuda")
    layers = [sr.LayerTensors(**vars(ns)) for ns in dev.layers]
    n_seg = len(wl.seg_lens)
    stream = torch.cuda.current_stream()

    def step():
        sr.replay_state(wl.shape, layers, n_seg, wl.t_total, dev.cu_seqlens, dev.slot_ids, ws, ws_bytes, stream)

    log(f"T={wl.t_total} rows x {len(wl.layers)} layers, workspace {ws_bytes / 2**20:.1f} MiB; warmup {args.warmup}")
    warm_run = warm_up(step, args.warmup)
    log(f"{warm_run} warmup steps run")

    ms_per_step, wall_ms, kt_all, dom = timed_steps(step, args.steps, stream)

    tokens = wl.replayed_tokens
    value = tokens / (ms_per_step / 1e3)
    log(f"{ms_per_step:.3f} ms/step (wall {wall_ms:.3f}), {value / 1e6:.2f} M tokens/s")

    work = algorithmic_work(wl, with_q=dev.with_q)
    kernels = {}
    total_all = max(sum(v[0] for v in kt_all.values()), 1e-12)
    for k, (tot, n) in kt_all.items():
        if n == 0:
            continue
        bound, amount = work[k]
        launches = n / BREAKDOWN_STEPS
        avg_ms = tot / n
        if bound == "mfma":
            dt = "f32" if wl.shape.anchor_dtype == "f32" else "bf16"
            ach, peak, unit = amount / (avg_ms * 1e-3) / 1e12, PEAK_TFLOPS[dt], "TFLOP/s"
        else:
            ach, peak, unit = amount / (avg_ms * 1e-3) / 1e9, PEAK_HBM_GBS, "GB/s"
        kernels[k] = {"avg_ms": round(avg_ms, 5), "launches_per_step": launches,
                      "share": round(kt_all[k][0] / total_all, 4),
                      "bound": bound, "achieved": round(ach, 2), "peak": peak, "unit": unit,
                      "frac": round(ach / peak, 4)}
    d = kernels[dom]
    traffic = measured_traffic(wl.name, dom)
    roofline = {"bound": d["bound"], "achieved": d["achieved"], "peak": d["peak"], "unit": d["unit"],
                "frac": d["frac"], "traffic": traffic, "kernel": dom}

    cpu = None
    if not args.no_cpu_baseline:
        log("timing the fp64 oracle on a bounded sample")
        cpu = cpu_baseline(wl, args.cpu_budget_s)

    sh = wl.shape
    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "warmup_run": warm_run, "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32" if sh.anchor_dtype == "f32" else "bf16",
        "data": "synthetic",
        "config": {"workload": wl.name, "requests": n_seg, "layers": len(wl.layers), "t_total": wl.t_total,
                   "replayed_tokens_per_step": tokens, "d_model": sh.d_model, "n_k_heads": sh.n_k_heads,
                   "n_v_heads": sh.n_v_heads, "d_k": sh.d_k, "d_v": sh.d_v, "conv_width": sh.conv_width,
                   "anchor_dtype": sh.anchor_dtype, "weight_dtype": sh.weight_dtype, "state_dtype": "f32"},
        "latency_ms": round(ms_per_step, 4),
        "roofline": roofline,
        "kernels": kernels,
        "kernels_timing": kernels_timing_note(dom),
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
