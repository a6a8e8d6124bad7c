#!/usr/bin/env python3
"""Throughput and latency of the COLD scoring path on one MI355X.

One step = one cold_score call over the whole batch of the serving-shaped
workload (32 requests x 2,000 candidate ads = 64,000 rows, 48 fields of dim
16 over 1M-row bf16 tables, SE block, 768x1024x512x256x128x64x2 network),
inputs resident in HBM before timing starts.  Prints one JSON line.

Also measured: per-stage kernel times with HIP events on the scoring stream
(a second pass of the same steps) and the roofline fraction of the dominant
kernel; the p50/p99 host-side latency of scoring one 2,000-ad request (eager
launches and HIP-graph replay); serving curves (one call over B requests,
and single requests replayed on K concurrent streams); the per-request
top-n selection by eCPM; and the CPU checker's throughput on a bounded
sample of the same workload.
"""
from __future__ import annotations

import argparse
import dataclasses
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
CSRC = os.path.join(ROOT, "paper_2007_16122_amd", "csrc")
TRAFFIC_JSON = os.path.join(ROOT, "profiles", "traffic_{workload}.json")
PEAK_MFMA_TFLOPS = {"bf16": 2500.0, "f16": 2500.0, "f32": 157.3}


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def stage_work(cfg, batch, stage, compact=False):
    """Algorithmic work of one launch of a stage: ('hbm', bytes) or
    ('mfma', flops). compact: the top-k model's network input keeps only
    each request's k groups (the first layer runs on k * d inputs; the
    call has an apply_compact stage)."""
    es = {"f32": 4, "bf16": 2, "f16": 2}[cfg.dtype]
    idb = 8 if cfg.hashed else 4
    R, Q = batch["n_rows"], len(batch["req_off"]) - 1
    d, m = cfg.emb_dim, cfg.n_groups
    nus = cfg.n_user + cfg.n_seq
    nax = cfg.n_ad + cfg.n_cross
    if stage == "user_pool":
        seq = int(batch["seq_off"][-1]) if cfg.n_seq else 0
        return "hbm", Q * cfg.n_user * (idb + d * es) + seq * (idb + d * es) + Q * nus * d * 4
    if stage in ("gather_se", "gather_apply", "se_weights"):
        # ids + gathered ad/cross rows + network input written + pooled user rows
        out = R * cfg.d_in * es if stage != "se_weights" else R * m * 4
        return "hbm", R * nax * (idb + d * es) + out + Q * nus * d * 4
    if stage == "gather_sq":
        # ids + gathered rows + the rows written exact (the input's place) + squeeze written
        return "hbm", R * nax * (idb + d * es) + R * cfg.d_in * es + R * m * 4 + Q * nus * d * 4
    if stage == "se_rows":      # squeeze read, SE weights written
        return "hbm", 2 * R * m * 4
    kin = min(cfg.topk_k, m) * d if compact else cfg.d_in   # width of the network input
    if stage == "apply":        # rows read and written in place, SE weights read
        return "hbm", 2 * R * cfg.d_in * es + R * m * 4
    if stage == "apply_compact":
        # kept groups read, compacted rows written, SE weights read; each
        # request's columns of the first layer's weights read and written
        return "hbm", 2 * R * kin * es + R * m * 4 + 2 * Q * cfg.widths[1] * kin * es
    if stage == "gather_raw":
        # ids + gathered ad/cross rows + the fp32 concatenated embedding written
        return "hbm", R * nax * (idb + d * es) + R * cfg.d_in * 4 + Q * nus * d * 4
    if stage == "se_dense":
        return "mfma_f32", 2.0 * R * cfg.d_in * m
    if stage == "dense_tail":     # the last separate layer and the fused tail
        w = cfg.widths
        return "mfma", 2.0 * R * (w[-5] * w[-4] + w[-4] * w[-3] + w[-3] * w[-2] + w[-2] * w[-1])
    if stage.startswith("dense"):
        li = int(stage[5:])
        k_in = kin if li == 0 else cfg.widths[li]
        return "mfma", 2.0 * R * k_in * cfg.widths[li + 1]
    if stage == "tail":
        w = cfg.widths
        return "mfma", 2.0 * R * (w[-4] * w[-3] + w[-3] * w[-2] + w[-2] * w[-1])
    if stage == "head":
        k = cfg.widths[-2]
        return "hbm", R * k * es + R * 4
    if stage == "group_mask":
        return "hbm", R * m * 4
    return "hbm", 0


def roofline_entry(cfg, batch, stage, ms, compact=False):
    kind, work = stage_work(cfg, batch, stage, compact)
    if kind in ("mfma", "mfma_f32"):
        ach = work / (ms * 1e-3) / 1e12
        peak = PEAK_MFMA_TFLOPS["f32" if kind == "mfma_f32" else cfg.dtype]
        return {"bound": "mfma", "achieved": round(ach, 2), "peak": peak, "unit": "TFLOP/s",
                "frac": round(ach / peak, 4), "work_per_launch": work}
    ach = work / (ms * 1e-3) / 1e9
    return {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": round(ach / PEAK_HBM_GBS, 4), "work_per_launch": work}


def request_slice(batch, q, cfg, q_end=None):
    """Requests q .. q_end-1 (default: request q alone) of a batch as a
    batch of their own (numpy)."""
    q_end = q + 1 if q_end is None else q_end
    off = batch["req_off"]
    lo, hi = int(off[q]), int(off[q_end])
    Q = len(off) - 1
    out = dict(req_off=(off[q:q_end + 1] - lo).astype(np.int32),
               user_ids=np.ascontiguousarray(batch["user_ids"][:, q:q_end]),
               ad_ids=np.ascontiguousarray(batch["ad_ids"][:, lo:hi]),
               cross_ids=np.ascontiguousarray(batch["cross_ids"][:, lo:hi]),
               n_rows=hi - lo, n_requests=q_end - q)
    if cfg.n_seq:
        so = batch["seq_off"]
        segs = [batch["seq_ids"][so[f * Q + qq]:so[f * Q + qq + 1]]
                for f in range(cfg.n_seq) for qq in range(q, q_end)]
        out["seq_off"] = np.concatenate([[0], np.cumsum([len(s) for s in segs])]).astype(np.int32)
        out["seq_ids"] = np.concatenate(segs)
    else:
        out["seq_off"] = np.zeros(1, np.int32)
        out["seq_ids"] = np.zeros(0, batch["ad_ids"].dtype)
    return out


def batching_curve(model, batch, cfg, sizes, iters, torch, binding):
    """Latency of one cold_score call over B requests of the batch (host
    wall clock to stream synchronisation) and the request rate a server that
    batches B requests per call would reach: B / p50."""
    out = []
    n_req = len(batch["req_off"]) - 1
    for b in sizes:
        if b > n_req:
            continue
        sub = binding.batch_to_device(request_slice(batch, 0, cfg, b), model.device)
        sc = torch.empty(max(sub["n_rows"], 1), dtype=torch.float32, device=model.device)
        p50, p99 = latency(model, sub, sc, iters, torch, graph=False)
        out.append({"requests_per_call": b, "p50_ms": round(p50, 4), "p99_ms": round(p99, 4),
                    "requests_per_s": round(b / (p50 * 1e-3), 1)})
        log(f"batching {b:2d} requests per call: p50 {p50:.4f} ms, p99 {p99:.4f} ms, "
            f"{out[-1]['requests_per_s']:.0f} req/s")
    return out


def gather_reference(cfg, batch, tables, iters, torch, dev):
    """Context for the gather's ceiling, not part of the scoring path: the
    table rows one scoring call reads (every group of every row, users' rows
    per request), gathered into the same [rows, groups, dim] layout with no
    SE block and no reweighting, from the tables laid end to end (each
    table's rows keep their positions), by
      - the plainest gather kernel (libcold_probe.so, include/cold_probe.h:
        int64 indices, two threads per row each copying 16 bytes, coalesced
        index reads and stores), which times the scattered row reads on
        their own, and
      - the vendor's generic gather, torch.index_select.
    Models with direct ids, 32-byte rows and no sequence or GPU-built cross
    groups only."""
    import ctypes
    from paper_2007_16122_amd import build as hip_build
    if cfg.hashed or cfg.n_seq or cfg.cross_pairs or cfg.emb_dim * (4 if cfg.dtype == "f32" else 2) != 32:
        return None
    R, V = batch["n_rows"], cfg.vocab
    off = torch.from_numpy(batch["req_off"].astype(np.int64)).to(dev)
    q_of_row = torch.repeat_interleave(torch.arange(len(off) - 1, device=dev), off[1:] - off[:-1])

    def col(ids, g):
        return torch.from_numpy(np.ascontiguousarray(ids).astype(np.int64)).to(dev) + g * V

    cols = [col(batch["user_ids"][f], f)[q_of_row] for f in range(cfg.n_user)]
    cols += [col(batch["ad_ids"][f], cfg.n_user + f) for f in range(cfg.n_ad)]
    cols += [col(batch["cross_ids"][f], cfg.n_user + cfg.n_ad + f) for f in range(cfg.n_cross)]
    idx = torch.stack(cols, dim=1).reshape(-1).contiguous()
    big = torch.cat(tables, 0)
    want = torch.index_select(big, 0, idx)
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def timed(fn):
        for _ in range(3):
            fn()
        e0.record(stream)
        for _ in range(iters):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / iters * 1e3

    out = torch.empty_like(want)
    vendor_us = timed(lambda: torch.index_select(big, 0, idx, out=out))
    probe_us = None
    if os.path.exists(hip_build.PROBE_LIB):
        plib = ctypes.CDLL(hip_build.PROBE_LIB)
        plib.cold_probe_row_gather.restype = ctypes.c_int
        plib.cold_probe_row_gather.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                                               ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]
        args = (big.data_ptr(), big.shape[0], idx.data_ptr(), out.data_ptr(), idx.numel(),
                stream.cuda_stream)
        out.zero_()

        def run():
            rc = plib.cold_probe_row_gather(*args)
            if rc != 0:
                raise RuntimeError(f"cold_probe_row_gather returned {rc}")

        probe_us = timed(run)
        if not torch.equal(out, want):
            raise RuntimeError("the row-gather probe does not reproduce torch.index_select")
    row_bytes = cfg.emb_dim * big.element_size()
    del big, out, idx, want
    return {"what": "the same table rows gathered into the same [rows, groups, dim] layout "
                    "with no SE and no reweighting; context only",
            "rows_gathered": R * cfg.n_groups,
            "rows_and_output_bytes": 2 * R * cfg.n_groups * row_bytes,
            "probe_us": None if probe_us is None else round(probe_us, 2),
            "vendor_index_select_us": round(vendor_us, 2)}


def time_workload(name, steps, warmup, torch, binding, synth, dev):
    """One other workload, timed the way the main one is: inputs resident,
    `warmup` untimed calls, then `steps` calls between two events with
    nothing recorded between the kernels, and a second pass with an event
    before every kernel stage for the per-stage times and rooflines."""
    cfg = synth.CONFIGS[name]
    batch = synth.make_batch(cfg, device=dev)
    params = synth.make_params(cfg)
    tables = [synth.table_torch(cfg, g, device=dev) for g in range(cfg.n_groups)]
    model = binding.ColdModel(cfg, device=dev)
    try:
        model.load(tables, binding.params_to_device(params, cfg.dtype, dev))
        dev_batch = binding.batch_to_device(batch, dev)
        R = batch["n_rows"]
        scores = torch.empty(R, dtype=torch.float32, device=dev)
        model.ensure_workspace(R, len(batch["req_off"]) - 1)
        for _ in range(warmup):
            model.score(dev_batch, scores=scores)
        torch.cuda.synchronize()
        assert bool(torch.isfinite(scores).all()), f"non-finite scores ({name})"
        stream = torch.cuda.current_stream()
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ev0.record(stream)
        for _ in range(steps):
            model.score(dev_batch, scores=scores)
        ev1.record(stream)
        torch.cuda.synchronize()
        ms = ev0.elapsed_time(ev1) / steps
        binding.cold_profile_enable(model.h, True)
        for _ in range(steps):
            model.score(dev_batch, scores=scores)
        torch.cuda.synchronize()
        stages, n_calls = binding.cold_profile_read(model.h)
        binding.cold_profile_enable(model.h, False)
    finally:
        model.close()
    compact = any(st == "apply_compact" for st, _ in stages)
    rows = []
    for st, tot in stages:
        e = roofline_entry(cfg, batch, st, tot / max(n_calls, 1), compact)
        e.update(name=st, ms=tot / max(n_calls, 1))
        rows.append(e)

    def frac(bound):
        part = [e for e in rows if e["bound"] == bound and not (bound == "hbm" and e["name"] == "head")]
        t = sum(e["ms"] for e in part)
        if not part or t <= 0:
            return None
        peak = part[0]["peak"] if bound == "hbm" else PEAK_MFMA_TFLOPS[cfg.dtype]
        scale = 1e9 if bound == "hbm" else 1e12
        return round(sum(e["work_per_launch"] for e in part) / (t * 1e-3) / scale / peak, 4)

    out = {"workload": name, "rows": R, "dtype": cfg.dtype, "steps": steps,
           "ms_per_step": round(ms, 5), "value": round(R / (ms * 1e-3), 1), "unit": "ads/s",
           "stages_us": {e["name"]: round(e["ms"] * 1e3, 2) for e in rows},
           "gather_se_hbm_frac": frac("hbm"), "mlp_mfma_frac": frac("mfma")}
    log(f"{name}: {ms:.4f} ms/step, {out['value']:.4g} ads/s, stages {out['stages_us']}")
    return out


def latency(model, dev_batch, scores, iters, torch, graph):
    stream = torch.cuda.current_stream()
    times = []
    if graph:
        g = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            model.score(dev_batch, scores=scores)
        stream.wait_stream(side)
        torch.cuda.synchronize()
        with torch.cuda.graph(g):
            model.score(dev_batch, scores=scores)
        g.replay()
        torch.cuda.synchronize()
        for _ in range(iters):
            t0 = time.perf_counter()
            g.replay()
            stream.synchronize()
            times.append(time.perf_counter() - t0)
    else:
        # a serving loop's call: buffers fixed, the call prepared once
        call = model.prepare(dev_batch, scores)
        for _ in range(iters):
            t0 = time.perf_counter()
            call()
            stream.synchronize()
            times.append(time.perf_counter() - t0)
    t = np.array(times) * 1e3
    return float(np.median(t)), float(np.quantile(t, 0.99))


def launch_sync_floor(torch, dev, iters):
    """p50 host time of launching one trivial kernel (a one-element add) on
    the current stream and synchronising it: the part of a request's latency
    that no kernel work can remove."""
    stream = torch.cuda.current_stream()
    t = torch.zeros(1, device=dev)
    for _ in range(10):
        t.add_(1)
    stream.synchronize()
    times = []
    for _ in range(iters):
        t0 = time.perf_counter()
        t.add_(1)
        stream.synchronize()
        times.append(time.perf_counter() - t0)
    return float(np.median(np.array(times) * 1e3))


def serving_curve(model, batch, cfg, streams, iters, torch, binding):
    """Concurrent serving of single requests: K streams, each replaying a HIP
    graph of one request's cold_score call back to back with its own
    workspace (the in-process analogue of the paper's MPS setup, Section 3.3).
    Per K: requests/s over the whole run and the per-request GPU latency
    (events around each replay) p50 / p99."""
    out = []
    n_req = len(batch["req_off"]) - 1
    for k in streams:
        ss = [torch.cuda.Stream() for _ in range(k)]
        graphs, keep = [], []
        for i, st in enumerate(ss):
            req = binding.batch_to_device(request_slice(batch, i % n_req, cfg), model.device)
            ws = torch.empty(max(binding.cold_workspace_bytes(model.h, req["n_rows"], 1), 256),
                             dtype=torch.uint8, device=model.device)
            sc = torch.empty(req["n_rows"], dtype=torch.float32, device=model.device)
            g = torch.cuda.CUDAGraph()
            st.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(st):
                model.score(req, scores=sc, workspace=ws)      # warm-up outside the graph
            torch.cuda.synchronize()
            with torch.cuda.graph(g, stream=st):
                model.score(req, scores=sc, workspace=ws)
            graphs.append(g)
            keep.append((req, ws, sc))
        torch.cuda.synchronize()
        ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(iters)] for _ in range(k)]
        for i in range(k):                                     # one untimed round
            with torch.cuda.stream(ss[i]):
                graphs[i].replay()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for it in range(iters):
            for i in range(k):
                with torch.cuda.stream(ss[i]):
                    ev[i][it][0].record(ss[i])
                    graphs[i].replay()
                    ev[i][it][1].record(ss[i])
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        lat = np.array([a.elapsed_time(b) for row in ev for a, b in row])
        out.append({"streams": k, "requests_per_s": round(k * iters / wall, 1),
                    "ads_per_s": round(k * iters * cfg.cand_per_request / wall, 1),
                    "p50_ms": round(float(np.median(lat)), 4),
                    "p99_ms": round(float(np.quantile(lat, 0.99)), 4)})
        log(f"serving {k:2d} streams: {out[-1]['requests_per_s']:9.1f} req/s, "
            f"p50 {out[-1]['p50_ms']:.4f} ms, p99 {out[-1]['p99_ms']:.4f} ms")
        del graphs, keep
    return out


def serving_worker(args):
    """One serving process of the multi-process measurement: builds the
    serving model on cuda:0, captures one 2,000-ad request's scoring call in
    a HIP graph, prints 'ready', waits for the start file, then replays the
    request back to back (one request in flight, host-side latency from
    replay to stream synchronisation) for the given time and prints one JSON
    line of latencies."""
    import torch
    from paper_2007_16122_amd import binding, synth
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    cfg = synth.CONFIGS[args.workload]
    batch = synth.make_batch(cfg, device=dev)
    params = synth.make_params(cfg)
    tables = [synth.table_torch(cfg, g, device=dev) for g in range(cfg.n_groups)]
    model = binding.ColdModel(cfg, device=dev)
    model.load(tables, binding.params_to_device(params, cfg.dtype, dev))
    q = args.worker_id % (len(batch["req_off"]) - 1)
    req = binding.batch_to_device(request_slice(batch, q, cfg), dev)
    sc = torch.empty(req["n_rows"], dtype=torch.float32, device=dev)
    ws = model.ensure_workspace(req["n_rows"], 1)
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(stream):
        for _ in range(3):
            model.score(req, scores=sc, workspace=ws)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        model.score(req, scores=sc, workspace=ws)
    lat = []
    with torch.cuda.stream(stream):   # replays go to the current stream
        for _ in range(20):
            g.replay()
        torch.cuda.synchronize()
        print("ready", flush=True)
        while not os.path.exists(args.start_file):
            time.sleep(0.0005)
        t_end = time.perf_counter() + args.duration
        while True:
            t0 = time.perf_counter()
            if t0 >= t_end:
                break
            g.replay()
            stream.synchronize()
            lat.append(time.perf_counter() - t0)
    torch.cuda.synchronize()
    print(json.dumps({"worker": args.worker_id, "requests": len(lat), "seconds": args.duration,
                      "lat_ms": [round(v * 1e3, 4) for v in lat]}), flush=True)
    del g
    model.close()


def serving_processes(args):
    """Concurrent serving from several processes on the one GPU (the analogue
    of the paper's CUDA MPS setup, Section 3.3, and of its usable-QPS
    measurement, Table 5): for each process count P, P workers each replay a
    graph of one 2,000-ad request back to back for the same interval; the
    aggregate request rate and the latency percentiles over all requests.
    The coordinating process never touches the GPU."""
    import subprocess
    import tempfile
    out = []
    for n_proc in [int(v) for v in args.serving_processes.split(",") if v]:
        start = os.path.join(tempfile.mkdtemp(prefix="cold_serve_"), "start")
        procs = [subprocess.Popen([sys.executable, os.path.abspath(__file__), "--serving-worker",
                                   "--worker-id", str(i), "--workload", args.workload,
                                   "--duration", str(args.duration), "--start-file", start],
                                  stdout=subprocess.PIPE, text=True)
                 for i in range(n_proc)]
        for p in procs:
            line = p.stdout.readline().strip()
            if line != "ready":
                for q in procs:
                    q.kill()
                raise RuntimeError(f"serving worker did not start: {line!r}")
        open(start, "w").close()
        results = []
        for p in procs:
            text, _ = p.communicate(timeout=args.duration + 120)
            if p.returncode != 0:
                raise RuntimeError(f"serving worker failed ({p.returncode})")
            results.append(json.loads(text.strip().splitlines()[-1]))
        lat = np.concatenate([np.asarray(r["lat_ms"]) for r in results])
        n_req = int(sum(r["requests"] for r in results))
        e = {"processes": n_proc, "requests_per_s": round(n_req / args.duration, 1),
             "ads_per_s": round(n_req * 2000 / args.duration, 1),
             "p50_ms": round(float(np.median(lat)), 4),
             "p99_ms": round(float(np.quantile(lat, 0.99)), 4),
             "requests": n_req}
        out.append(e)
        log(f"serving {n_proc:2d} processes: {e['requests_per_s']:9.1f} req/s, p50 {e['p50_ms']:.4f} ms, "
            f"p99 {e['p99_ms']:.4f} ms")
    usable = {f"p99<={lim}ms": max([e["requests_per_s"] for e in out if e["p99_ms"] <= lim],
                                   default=None) for lim in (0.1, 0.25, 0.5, 1.0)}
    print(json.dumps({"workload": args.workload, "duration_s": args.duration,
                      "serving_processes": out, "usable_requests_per_s": usable}), flush=True)


def groups_sweep(base, counts, steps, warmup, torch, binding, synth, dev):
    """Throughput of lightweight models that keep K feature groups (Section
    3.2, feature group selection: the offline tests weigh a model with the
    top-K groups by GAUC, QPS and RT).  Each K gets a model of its own with
    K groups split 1:2:1 over user, ad and cross fields and the serving
    batch shape; only its speed is measured (synthetic weights)."""
    out = []
    for k in counts:
        nu, nx = k // 4, k // 4
        cfg = dataclasses.replace(base, n_user=nu, n_ad=k - nu - nx, n_cross=nx, n_seq=0,
                                  topk_k=0, emit_importance=False,
                                  widths=(k * base.emb_dim,) + tuple(base.widths[1:]))
        batch = synth.make_batch(cfg, device=dev)
        tables = [synth.table_torch(cfg, g, device=dev) for g in range(cfg.n_groups)]
        model = binding.ColdModel(cfg, device=dev)
        model.load(tables, binding.params_to_device(synth.make_params(cfg), cfg.dtype, dev))
        dev_batch = binding.batch_to_device(batch, dev)
        scores = torch.empty(batch["n_rows"], dtype=torch.float32, device=dev)
        for _ in range(warmup):
            model.score(dev_batch, scores=scores)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(steps):
            model.score(dev_batch, scores=scores)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / steps
        out.append({"groups": k, "d_in": cfg.d_in, "ms_per_step": round(ms, 5),
                    "ads_per_s": round(batch["n_rows"] / (ms * 1e-3), 1)})
        log(f"groups {k:4d} (D_in {cfg.d_in:5d}): {ms:.4f} ms/step, {out[-1]['ads_per_s']:.4g} ads/s")
        model.close()
        del tables, model, dev_batch, scores
        torch.cuda.empty_cache()
    return out


def cpu_baseline(cfg, batch, params, target_s, gpu_scores=None, one_core_s=0.0):
    """The CPU checker, as it stands, on a bounded sample of the workload;
    with `gpu_scores` (the GPU's scores of the whole batch) also the
    |GPU - checker| CTR statistics over the sampled rows, and with
    `one_core_s` > 0 the checker's rate on one thread over a smaller
    sample."""
    import oracle
    from paper_2007_16122_amd import synth
    dims = dict(n_user=cfg.n_user, n_seq=cfg.n_seq, n_ad=cfg.n_ad, n_cross=cfg.n_cross,
                emb_dim=cfg.emb_dim, se_hidden=cfg.se_hidden, dtype=cfg.dtype,
                hashed=cfg.hashed, linear_log=cfg.linear_log, topk_k=cfg.topk_k,
                widths=list(cfg.widths), cross_pairs=[list(p) for p in cfg.cross_pairs])
    stored = dict(params)
    stored["mlp_w"] = [synth.mlp_weight_stored(w, cfg.dtype) for w in params["mlp_w"]]
    np_dt = {"f32": np.float32, "f16": np.float16, "bf16": np.uint16}[cfg.dtype]

    def tables_for(sample):
        q_n = len(batch["req_off"]) - 1
        reqs = np.unique(np.searchsorted(batch["req_off"], sample, side="right") - 1)
        tabs = []
        for g in range(cfg.n_groups):
            kind = cfg.group_kind(g)
            if kind == "user":
                ids = batch["user_ids"][g][reqs]
            elif kind == "seq":
                f = g - cfg.n_user
                so = batch["seq_off"]
                ids = np.concatenate([batch["seq_ids"][so[f * q_n + q]:so[f * q_n + q + 1]]
                                      for q in reqs])
            elif kind == "ad":
                ids = batch["ad_ids"][g - cfg.n_user - cfg.n_seq][sample]
            elif cfg.cross_pairs:
                uf, af = cfg.cross_pairs[g - cfg.n_user - cfg.n_seq - cfg.n_ad]
                width = (1 << 64) - 1 if cfg.hashed else (1 << 32) - 1
                req_of = np.searchsorted(batch["req_off"], sample, side="right") - 1
                pairs = set(zip((int(v) & width for v in batch["user_ids"][uf][req_of]),
                                (int(v) & width for v in batch["ad_ids"][af][sample])))
                ids = None
                rows = np.unique(np.array([oracle.hash_row(oracle.cross_key(u, a), g, cfg.vocab)
                                           for u, a in pairs], np.int64))
            else:
                ids = batch["cross_ids"][g - cfg.n_user - cfg.n_seq - cfg.n_ad][sample]
            if ids is not None:
                rows = (np.array([oracle.hash_row(int(v), g, cfg.vocab) for v in np.unique(ids)])
                        if cfg.hashed else np.unique(ids)).astype(np.int64)
            t = np.zeros((cfg.vocab, cfg.emb_dim), np_dt)
            t[rows] = synth.table_rows_numpy(cfg, g, rows)
            tabs.append(t)
        return tabs

    threads = len(os.sched_getaffinity(0))
    probe = np.arange(min(128, batch["n_rows"]))
    tabs = tables_for(probe)
    t0 = time.perf_counter()
    oracle.score(dims, tabs, stored, batch, sample=probe, n_threads=threads)
    per_row = (time.perf_counter() - t0) / len(probe)
    n = int(min(batch["n_rows"], max(len(probe), target_s / max(per_row, 1e-9))))
    sample = np.arange(n)
    tabs = tables_for(sample)
    t0 = time.perf_counter()
    o = oracle.score(dims, tabs, stored, batch, sample=sample, n_threads=threads)
    dt = time.perf_counter() - t0
    out = {"value": round(n / dt, 1), "unit": "ads/s", "cores": int(o["n_threads"]),
           "kind": "oracle", "seconds": round(dt, 2),
           "sample": f"first {n} rows (requests 0..{int(np.searchsorted(batch['req_off'], n - 1, side='right')) - 1}) "
                     f"of the {cfg.name} batch, fp64 checker, {o['n_threads']} threads"}
    parity = None
    if gpu_scores is not None:
        d = np.abs(np.asarray(gpu_scores, np.float64)[sample] - o["scores"])
        tol = 1e-5 if cfg.dtype == "f32" else 2e-3
        parity = {"rows": int(n), "max_abs_dctr": float(d.max()),
                  "p99_abs_dctr": float(np.quantile(d, 0.99)), "mean_abs_dctr": float(d.mean()),
                  "tol": tol, "within_tol": bool(d.max() <= tol),
                  "ctr_mean": float(o["scores"].mean()), "ctr_std": float(o["scores"].std())}
    one = None
    if one_core_s > 0:
        n1 = int(min(n, max(len(probe), one_core_s / max(per_row * threads, 1e-9))))
        t0 = time.perf_counter()
        oracle.score(dims, tabs, stored, batch, sample=np.arange(n1), n_threads=1)
        dt1 = time.perf_counter() - t0
        one = {"value": round(n1 / dt1, 1), "unit": "ads/s", "cores": 1, "kind": "oracle",
               "seconds": round(dt1, 2), "sample": f"first {n1} rows, one thread"}
    return out, parity, one


# ---------------------------------------------------------------------------
# rocprofv3 post-processing (runs on the host after a profiled bench run)
def _source_hashes():
    import hashlib
    out = {}
    for name in sorted(os.listdir(CSRC)):
        if name.endswith((".hip", ".h")):
            with open(os.path.join(CSRC, name), "rb") as fh:
                out[name] = hashlib.sha256(fh.read()).hexdigest()
    return out


def _stage_of(kernel_name, dense_index):
    """Stage name of one of our kernels, in cold_score's launch order."""
    if "user_pool" in kernel_name:
        return "user_pool"
    if "gather_se_kernel" in kernel_name:
        # the second template argument (mangled "Li<n>E") is the pass:
        # full, weights, apply, raw
        mt = re.search(r"gather_se_kernelI\w*?Li(\d+)E", kernel_name)
        mode = mt.group(1) if mt else "0"
        return {"0": "gather_se", "1": "se_weights", "2": "gather_apply", "3": "gather_raw",
                "4": "gather_sq"}.get(mode, "gather_se")
    if "gather_full" in kernel_name:
        return "gather_se"
    if "se_rows_kernel" in kernel_name:
        return "se_rows"
    if "apply_weights_kernel" in kernel_name:
        return "apply"
    if "apply_compact_kernel" in kernel_name:
        return "apply_compact"
    if "dense_f32" in kernel_name:
        return "se_dense"
    if "dense_tail_kernel" in kernel_name:
        return "dense_tail"
    if "mask_partial" in kernel_name or "mask_select" in kernel_name:
        return "group_mask"
    if "dense_relu" in kernel_name:
        return f"dense{dense_index}"
    if "mlp_tail" in kernel_name:
        return "tail"
    if "head_kernel" in kernel_name:
        return "head"
    return None


def _ours(rows):
    """Dispatches of libcold kernels in launch order. rocprofv3 prints some
    kernel names mangled and some demangled, so both forms are matched."""
    ours = [r for r in rows if ("4cold" in r["Kernel_Name"] or "cold::" in r["Kernel_Name"])
            and "clear_flag" not in r["Kernel_Name"] and "transpose_f32" not in r["Kernel_Name"]
            and "pack_frag" not in r["Kernel_Name"]]
    ours.sort(key=lambda r: int(r["Start_Timestamp"]))
    return ours


def _label_call(call):
    """(stage, row) pairs of one scoring call. A demangled gather name does
    not carry its pass; the gather right before the group mask is the
    importance pass."""
    out, di = [], 0
    for r in call:
        st = _stage_of(r["Kernel_Name"], di)
        # the fp32 matrix-core layer is the literal SE layer right after the
        # raw gather, and a hidden layer of an fp32 model anywhere else
        if st == "se_dense" and not (out and out[-1][0] == "gather_raw"):
            st = f"dense{di}"
        if st and st.startswith("dense"):
            di += 1
        out.append([st, r])
    for i in range(len(out) - 1):
        if out[i][0] == "gather_se" and out[i + 1][0] == "group_mask":
            out[i][0] = "se_weights"
        if out[i][0] == "gather_se" and out[i + 1][0] == "se_rows":
            out[i][0] = "gather_sq"
    return [tuple(x) for x in out]


def _call_starts(ours):
    """Indices of the first kernel of each scoring call: the per-request
    user pooling, or, in a call without one, the first gather after the
    previous call's last layer."""
    out, prev = [], None
    for i, r in enumerate(ours):
        st = _stage_of(r["Kernel_Name"], 0)
        if st == "user_pool" or (st in ("gather_se", "se_weights", "gather_raw", "gather_sq")
                                 and prev != "user_pool"):
            out.append(i)
        if st is not None:
            prev = st
    return out


def _last_call(rows, key_start="Start_Timestamp"):
    """Dispatches of libcold kernels in the last complete scoring call,
    as (stage, row) pairs in launch order."""
    ours = _ours(rows)
    starts = _call_starts(ours)
    if not starts:
        return []
    return _label_call(ours[starts[-1]:])


def summarize_single_request(trace_dir, command):
    """Per-kernel durations of the single-request scoring calls (the latency
    loops: one 2,000-ad request of the serving model) from a rocprofv3
    --kernel-trace CSV directory: median and 10th/90th percentiles per
    kernel, the gaps between consecutive kernels and the span of a call.
    A call starts at its pooling or gather kernel; calls of fewer than four
    kernels or with a kernel of more than 200,000 threads (the whole batch)
    are left out."""
    import csv
    import glob
    import statistics
    path = glob.glob(os.path.join(trace_dir, "**", "*kernel_trace.csv"), recursive=True)[0]
    rows = sorted((r for r in csv.DictReader(open(path)) if "cold" in r["Kernel_Name"]),
                  key=lambda r: int(r["Start_Timestamp"]))

    def short(n):
        for k, v in (("user_pool", "user_pool"), ("gather_full", "gather_se"),
                     ("gather_se", "gather_se"), ("dense_tail", "dense_tail"),
                     ("mlp_tail", "tail"), ("dense_relu_buf", "dense")):
            if k in n:
                return v
        return None

    calls, cur = [], []
    for r in rows:
        st = short(r["Kernel_Name"])
        if st is None:
            continue
        starts = st == "user_pool" or (st == "gather_se" and not (
            cur and short(cur[-1]["Kernel_Name"]) == "user_pool"))
        if starts and cur:
            calls.append(cur)
            cur = []
        cur.append(r)
    if cur:
        calls.append(cur)
    small = [c for c in calls if len(c) >= 4 and all(int(x["Grid_Size_X"]) <= 200000 for x in c)]
    if not small:
        return "no single-request calls in the trace\n"
    names = []
    for i, r in enumerate(small[0]):
        st = short(r["Kernel_Name"])
        if st == "dense":
            st = "dense%d" % sum(1 for x in small[0][:i] if short(x["Kernel_Name"]) == "dense")
        names.append(st)

    def us(a, b):
        return (int(a) - int(b)) / 1e3

    def pct(v, f):
        v = sorted(v)
        return v[min(len(v) - 1, int(f * len(v)))]

    out = ["# rocprofv3 kernel trace of single-request scoring calls (one 2,000-ad request "
           "of the serving model, bf16)",
           f"# command: {command}",
           "# calls: the eager and HIP-graph latency loops; a call = " + ", ".join(names)
           + " on 2,000 rows",
           f"# {len(small)} single-request calls",
           f"{'stage':12s} {'median_us':>9s} {'p10_us':>7s} {'p90_us':>7s}  grid  kernel"]
    for i, nm in enumerate(names):
        v = [us(c[i]["End_Timestamp"], c[i]["Start_Timestamp"]) for c in small if len(c) > i]
        out.append(f"{nm:12s} {statistics.median(v):9.2f} {pct(v, .1):7.2f} {pct(v, .9):7.2f}  "
                   f"{small[0][i]['Grid_Size_X']}  {small[0][i]['Kernel_Name'][:100]}")
    gaps = [statistics.median([us(c[i]["Start_Timestamp"], c[i - 1]["End_Timestamp"])
                               for c in small if len(c) > i]) for i in range(1, len(names))]
    out.append("gaps between consecutive kernels, median us: " + ", ".join(f"{g:.2f}" for g in gaps))
    out.append("first kernel start to last kernel end, median us: %.2f" % statistics.median(
        [us(c[-1]["End_Timestamp"], c[0]["Start_Timestamp"]) for c in small]))
    return "\n".join(out) + "\n"


def summarize_trace(trace_dir, command):
    """Per-stage kernel durations (mean over the profiled calls) from a
    rocprofv3 --kernel-trace CSV directory."""
    import csv
    import glob
    path = glob.glob(os.path.join(trace_dir, "**", "*kernel_trace.csv"), recursive=True)[0]
    rows = list(csv.DictReader(open(path)))
    ours = _ours(rows)
    starts = _call_starts(ours)
    per_stage = {}
    for a, b in zip(starts, starts[1:] + [len(ours)]):
        for st, r in _label_call(ours[a:b]):
            st = st or "other"
            d = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-3
            per_stage.setdefault(st, {"us": [], "kernel": r["Kernel_Name"], "grid": r.get("Grid_Size_X", r.get("Grid_Size", "?"))})["us"].append(d)
    lines = [f"# rocprofv3 kernel trace, per stage of one cold_score call", f"# command: {command}",
             f"# {len(starts)} calls profiled", f"{'stage':12s} {'calls':>5s} {'mean_us':>9s} {'min_us':>9s} {'max_us':>9s}  grid  kernel"]
    for st, v in per_stage.items():
        us = v["us"]
        lines.append(f"{st:12s} {len(us):5d} {np.mean(us):9.2f} {np.min(us):9.2f} {np.max(us):9.2f}  {v['grid']}  {v['kernel'][:90]}")
    return "\n".join(lines) + "\n"


def summarize_pmc(fetch_dir, write_dir, probe_mb, command, workload):
    """HBM bytes per launch of each stage from FETCH_SIZE and WRITE_SIZE runs,
    each scaled so that the plain copy probe of probe_mb MiB reads (writes)
    exactly probe_mb MiB."""
    import csv
    import glob
    res = {}
    for counter, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        path = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)[0]
        rows = [r for r in csv.DictReader(open(path)) if r["Counter_Name"] == counter]
        copies = [r for r in rows if "copyBuffer" in r["Kernel_Name"]]
        copies.sort(key=lambda r: int(r["Start_Timestamp"]))
        probe_kib = float(copies[-1]["Counter_Value"])      # the probe runs last
        factor = probe_mb * 1024.0 / probe_kib
        stages = {}
        for st, r in _last_call(rows):
            stages.setdefault(st, 0.0)
            stages[st] += float(r["Counter_Value"]) * factor * 1024.0
        res[counter] = {"factor": factor, "probe_raw_kib": probe_kib, "stages": stages}
    stages = {}
    for st in res["FETCH_SIZE"]["stages"]:
        stages[st] = {"fetch_bytes": round(res["FETCH_SIZE"]["stages"][st]),
                      "write_bytes": round(res["WRITE_SIZE"]["stages"].get(st, 0.0))}
    return {"workload": workload, "command": command, "probe_mb": probe_mb,
            "fetch_factor": res["FETCH_SIZE"]["factor"], "write_factor": res["WRITE_SIZE"]["factor"],
            "stages": stages, "sources": _source_hashes()}


def summarize_probe(fetch_dir, write_dir, probe_mb, command):
    """HBM bytes per dispatch of the row-gather probe (the gather's ceiling
    measurement) from FETCH_SIZE and WRITE_SIZE runs, scaled so that the
    plain copy of probe_mb MiB (the largest copy in the run) reads (writes)
    exactly probe_mb MiB; beside it the fused gather's bytes from the
    serving workload's traffic file."""
    import csv
    import glob
    import statistics
    out = {}
    for counter, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        path = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)[0]
        rows = [r for r in csv.DictReader(open(path)) if r["Counter_Name"] == counter]
        copy_kib = max(float(r["Counter_Value"]) for r in rows if "copyBuffer" in r["Kernel_Name"])
        factor = probe_mb * 1024.0 / copy_kib
        vals = [float(r["Counter_Value"]) * factor * 1024.0 for r in rows
                if "row_gather_probe_kernel" in r["Kernel_Name"]]
        out[counter] = (statistics.median(vals), len(vals), factor)
    fused = load_traffic("serving_bf16")
    fg = fused["stages"].get("gather_se") if fused else None
    f, w = out["FETCH_SIZE"][0], out["WRITE_SIZE"][0]
    lines = ["# rocprofv3 HBM traffic of the row-gather probe (libcold_probe.so) on the rows of one",
             "# scoring call of the serving workload (3,072,000 rows of 32 bytes gathered into the",
             "# [rows, groups, dim] layout; int64 indices), beside the fused gather+SE of the same call",
             f"# command: {command}",
             f"# FETCH_SIZE scaled by {out['FETCH_SIZE'][2]:.3f}, WRITE_SIZE by "
             f"{out['WRITE_SIZE'][2]:.3f} (the {probe_mb} MiB copy reads and writes {probe_mb} MiB);"
             f" median over {out['FETCH_SIZE'][1]} dispatches",
             f"{'kernel':28s} {'fetch_MB':>9s} {'write_MB':>9s} {'total_MB':>9s}",
             f"{'row_gather_probe':28s} {f / 1e6:9.1f} {w / 1e6:9.1f} {(f + w) / 1e6:9.1f}"]
    if fg:
        lines.append(f"{'gather_se (fused, profiles)':28s} {fg['fetch_bytes'] / 1e6:9.1f} "
                     f"{fg['write_bytes'] / 1e6:9.1f} {(fg['fetch_bytes'] + fg['write_bytes']) / 1e6:9.1f}")
    return "\n".join(lines) + "\n"


def summarize_mfma(pmc_dir, command, workload, simds, xcds):
    """Matrix-core utilisation per stage from one rocprofv3 run with
    SQ_VALU_MFMA_BUSY_CYCLES and GRBM_GUI_ACTIVE: the first summed over all
    SIMDs, the second over the XCDs, so busy = (MFMA busy cycles per SIMD) /
    (active cycles of the dispatch). It does not depend on the clock the
    chip ran at, unlike the achieved rate against the 2.5 PFLOP/s peak."""
    import csv
    import glob
    path = glob.glob(os.path.join(pmc_dir, "**", "*counter_collection.csv"), recursive=True)[0]
    rows = list(csv.DictReader(open(path)))
    val = {}
    for counter in ("SQ_VALU_MFMA_BUSY_CYCLES", "GRBM_GUI_ACTIVE"):
        for st, r in _last_call([r for r in rows if r["Counter_Name"] == counter]):
            val.setdefault(st, {}).setdefault(counter, 0.0)
            val[st][counter] += float(r["Counter_Value"])
            val[st]["kernel"] = r["Kernel_Name"]
    lines = [f"# rocprofv3 matrix-core utilisation, per stage of one cold_score call ({workload})",
             f"# command: {command}",
             f"# busy = SQ_VALU_MFMA_BUSY_CYCLES / {simds} SIMDs over GRBM_GUI_ACTIVE / {xcds} XCDs",
             f"{'stage':12s} {'mfma_busy_per_simd':>18s} {'active_cycles':>13s} {'busy':>6s}  kernel"]
    for st, v in val.items():
        busy = v.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0) / simds
        active = v.get("GRBM_GUI_ACTIVE", 0.0) / xcds
        frac = busy / active if active else float("nan")
        lines.append(f"{st:12s} {busy:18.0f} {active:13.0f} {frac:6.3f}  {v['kernel'][:90]}")
    return "\n".join(lines) + "\n"


def summarize_parity(run_dir, command):
    """profiles/parity_<workload>.txt from one GPU run: the |GPU - checker|
    CTR statistics of every parity test (the JSON lines the tests append to
    COLD_PARITY_LOG) and of the bench's checked sample (bench_<workload>.json)."""
    tests = {}
    path = os.path.join(run_dir, "parity.jsonl")
    if os.path.exists(path):
        for line in open(path):
            e = json.loads(line)
            if "max" in e:
                tests.setdefault(e["workload"], []).append(e)
    written = []
    names = sorted(set(tests) | {f[6:-5] for f in os.listdir(run_dir)
                                 if f.startswith("bench_") and f.endswith(".json")})
    for w in names:
        lines = [f"# |GPU - checker| CTR per parity check, workload {w}",
                 f"# command: {command}"]
        bj = os.path.join(run_dir, f"bench_{w}.json")
        if os.path.exists(bj):
            rows = [l for l in open(bj).read().splitlines() if l.startswith("{")]
            if rows:
                b = json.loads(rows[-1])
                p = b.get("parity")
                if p:
                    lines.append(f"# bench.py --workload {w}: full-size batch, the checked sample of "
                                 f"the CPU baseline leg ({b['cpu_baseline']['sample']})")
                    lines.append(f"{'check':52s} {'rows':>7s} {'max':>9s} {'p99':>9s} {'mean':>9s} "
                                 f"{'tol':>7s} {'ctr_mean':>8s} {'ctr_std':>8s}")
                    lines.append(f"{'bench full-size sample':52s} {p['rows']:7d} {p['max_abs_dctr']:9.2e} "
                                 f"{p['p99_abs_dctr']:9.2e} {p['mean_abs_dctr']:9.2e} {p['tol']:7.0e} "
                                 f"{p['ctr_mean']:8.4f} {p['ctr_std']:8.4f}")
        if w in tests:
            if len(lines) == 2:
                lines.append(f"{'check':52s} {'rows':>7s} {'max':>9s} {'p99':>9s} {'mean':>9s} "
                             f"{'tol':>7s} {'ctr_mean':>8s} {'ctr_std':>8s}")
            for e in tests[w]:
                lines.append(f"{e['label'][:52]:52s} {e['n']:7d} {e['max']:9.2e} {e['p99']:9.2e} "
                             f"{e['mean']:9.2e} {e['tol']:7.0e} {e['ctr_mean']:8.4f} {e['ctr_std']:8.4f}")
        out = os.path.join(ROOT, "profiles", f"parity_{w}.txt")
        with open(out, "w") as fh:
            fh.write("\n".join(lines) + "\n")
        written.append(out)
    return written


def _stage_sources(stage):
    """Source files that define a stage's kernel (with the shared header)."""
    if stage.startswith("dense") or stage in ("tail", "head", "se_dense"):
        return ("mlp.hip", "cold_internal.h")
    return ("gather.hip", "cold_internal.h")


def load_traffic(workload):
    """Measured HBM bytes per stage, keeping only the stages whose kernel
    sources are unchanged since the counters were taken (None if none are)."""
    path = TRAFFIC_JSON.format(workload=workload)
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        t = json.load(fh)
    then, now = t.get("sources", {}), _source_hashes()
    stages = {k: v for k, v in t.get("stages", {}).items()
              if all(then.get(f) is not None and then.get(f) == now.get(f) for f in _stage_sources(k))}
    return dict(t, stages=stages) if stages else None


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="serving_bf16")
    ap.add_argument("--latency-iters", type=int, default=300)
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-one-core-seconds", type=float, default=3.0,
                    help="also time the checker on one thread for about this long (0 = skip)")
    ap.add_argument("--copy-probe-mb", type=int, default=0,
                    help="after timing, copy this many MiB device-to-device once (a plain "
                         "copy of known size, to calibrate HBM byte counters)")
    ap.add_argument("--se-literal", action="store_true",
                    help="use the SE block of Eq. 2 as printed (one FC over the concatenated "
                         "embedding) instead of the squeeze/excitation form")
    ap.add_argument("--groups-sweep", default="",
                    help="after timing, the throughput of models keeping K groups, for each K "
                         "of this comma list (serving batch shape, widths of --workload)")
    ap.add_argument("--gpu-cross", action="store_true",
                    help="build every cross field on the GPU from a (user field, ad field) "
                         "id pair instead of reading per-row cross ids")
    ap.add_argument("--topn", type=int, default=200,
                    help="after timing, time the per-request top-n selection by eCPM "
                         "(0 = skip); not part of the timed step")
    ap.add_argument("--serving-streams", default="1,2,4,8,16",
                    help="after timing, concurrent single-request serving on this many streams "
                         "(comma list; empty = skip)")
    ap.add_argument("--serving-iters", type=int, default=200)
    ap.add_argument("--batching", default="1,2,4,8,16,32",
                    help="after timing, the latency of one call over this many requests "
                         "(comma list; empty = skip)")
    ap.add_argument("--no-latency", action="store_true",
                    help="skip every measurement after the timed steps: the 2,000-ad latency, "
                         "the serving curves and the top-n selection (kernel-trace profiles of "
                         "the step only)")
    ap.add_argument("--other-workloads",
                    default="tiny_fp32,multivalued_fp16_ll,large_fp16_ll,wide_prune_bf16",
                    help="comma-separated workloads also timed in the same run (step time, "
                         "stage times, rooflines) and listed under other_workloads; '' for none")
    ap.add_argument("--serving-processes", default="",
                    help="only measure concurrent serving from this many processes (comma list), "
                         "each replaying a 2,000-ad request back to back, and print one JSON line")
    ap.add_argument("--duration", type=float, default=2.0,
                    help="seconds of back-to-back requests per process count")
    ap.add_argument("--serving-worker", action="store_true", help=argparse.SUPPRESS)
    ap.add_argument("--worker-id", type=int, default=0, help=argparse.SUPPRESS)
    ap.add_argument("--start-file", default="", help=argparse.SUPPRESS)
    ap.add_argument("--summarize-trace", metavar="DIR",
                    help="print a per-stage summary of a rocprofv3 kernel-trace run and exit")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="write profiles/traffic_<workload>.json from FETCH_SIZE / WRITE_SIZE runs")
    ap.add_argument("--summarize-probe", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="summarise FETCH_SIZE/WRITE_SIZE runs of the row-gather probe and exit")
    ap.add_argument("--summarize-single-request", metavar="DIR",
                    help="summarise a kernel trace of the latency loops (single requests) and exit")
    ap.add_argument("--summarize-parity", metavar="DIR",
                    help="write profiles/parity_<workload>.txt from a GPU run's parity.jsonl "
                         "(tests with COLD_PARITY_LOG) and bench_<workload>.json files, and exit")
    ap.add_argument("--summarize-mfma", metavar="DIR",
                    help="print matrix-core utilisation per stage from a run with "
                         "--pmc SQ_VALU_MFMA_BUSY_CYCLES GRBM_GUI_ACTIVE")
    ap.add_argument("--simds", type=int, default=1024, help="SIMDs on the chip (MI355X: 256 CUs x 4)")
    ap.add_argument("--xcds", type=int, default=8, help="XCDs on the chip")
    ap.add_argument("--profile-command", default="", help="command recorded in summaries")
    args = ap.parse_args()
    if args.serving_worker:
        serving_worker(args)
        return
    if args.serving_processes:
        serving_processes(args)
        return
    if args.summarize_parity:
        for path in summarize_parity(args.summarize_parity, args.profile_command):
            print(path)
        return
    if args.summarize_trace:
        print(summarize_trace(args.summarize_trace, args.profile_command), end="")
        return
    if args.summarize_probe:
        print(summarize_probe(args.summarize_probe[0], args.summarize_probe[1],
                              args.copy_probe_mb or 1024, args.profile_command), end="")
        return
    if args.summarize_single_request:
        print(summarize_single_request(args.summarize_single_request, args.profile_command), end="")
        return
    if args.summarize_mfma:
        print(summarize_mfma(args.summarize_mfma, args.profile_command, args.workload, args.simds,
                             args.xcds), end="")
        return
    if args.summarize_pmc:
        t = summarize_pmc(args.summarize_pmc[0], args.summarize_pmc[1], args.copy_probe_mb or 1024,
                          args.profile_command, args.workload)
        path = TRAFFIC_JSON.format(workload=args.workload)
        with open(path, "w") as fh:
            json.dump(t, fh, indent=1)
        print(json.dumps(t["stages"], indent=1))
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: the scoring path runs on a single MI355X "
              f"(rows are independent, so it would shard by requests across GPUs). "
              f"Got --gpus {args.gpus}.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2007_16122_amd import binding, synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    cfg = synth.CONFIGS[args.workload]
    if args.se_literal:
        cfg = synth.config(cfg.name, se_form="literal")
    if args.gpu_cross:
        # every cross field built on the GPU from a (user field, ad field) pair
        cfg = synth.config(cfg.name, cross_pairs=tuple(
            (f % cfg.n_user, f % cfg.n_ad) for f in range(cfg.n_cross)))
    log(f"workload {cfg.name}: {cfg.n_requests} x {cfg.cand_per_request} rows, "
        f"{cfg.n_groups} groups, vocab {cfg.vocab}, {cfg.dtype}")
    t0 = time.perf_counter()
    batch = synth.make_batch(cfg, device=dev)
    params = synth.make_params(cfg)
    tables = [synth.table_torch(cfg, g, device=dev) for g in range(cfg.n_groups)]
    model = binding.ColdModel(cfg, device=dev)
    model.load(tables, binding.params_to_device(params, cfg.dtype, dev))
    dev_batch = binding.batch_to_device(batch, dev)
    R = batch["n_rows"]
    scores = torch.empty(R, dtype=torch.float32, device=dev)
    model.ensure_workspace(R, len(batch["req_off"]) - 1)
    torch.cuda.synchronize()
    log(f"inputs ready in {time.perf_counter() - t0:.1f}s")

    for _ in range(args.warmup):
        model.score(dev_batch, scores=scores)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(scores).all()), "non-finite scores"

    # timed region: K steps, nothing recorded between the kernels
    stream = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        model.score(dev_batch, scores=scores)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    ms_per_step = ev0.elapsed_time(ev1) / args.steps
    value = R / (ms_per_step * 1e-3)
    log(f"{args.steps} steps: {ms_per_step:.4f} ms/step (wall {wall * 1e3 / args.steps:.4f}), "
        f"{value:.4g} ads/s")
    # the same K steps again with a HIP event on the stream before every
    # kernel stage: per-kernel durations for the rooflines (an event between
    # two kernels stops the next one from starting early, so this pass is a
    # little slower than the one above)
    binding.cold_profile_enable(model.h, True)
    p0, p1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    p0.record(stream)
    for _ in range(args.steps):
        model.score(dev_batch, scores=scores)
    p1.record(stream)
    torch.cuda.synchronize()
    stages, n_calls = binding.cold_profile_read(model.h)
    binding.cold_profile_enable(model.h, False)
    ms_profiled = p0.elapsed_time(p1) / args.steps
    log(f"with stage events: {ms_profiled:.4f} ms/step")

    stage_rows = []
    compact = any(name == "apply_compact" for name, _ in stages)
    for name, tot in stages:
        ms = tot / max(n_calls, 1)
        e = roofline_entry(cfg, batch, name, ms, compact)
        e.update(name=name, ms=round(ms, 5))
        stage_rows.append(e)
        log(f"  {name:12s} {ms * 1e3:9.2f} us  {e['achieved']:>9} {e['unit']}  ({100 * e['frac']:.1f}%)")
    dom = max(stage_rows, key=lambda e: e["ms"])
    traffic = load_traffic(cfg.name)
    dom_traffic = None
    if traffic and dom["name"] in traffic["stages"]:
        tb = traffic["stages"][dom["name"]]
        dom_traffic = tb["fetch_bytes"] + tb["write_bytes"]
    roofline = {"bound": dom["bound"], "achieved": dom["achieved"], "peak": dom["peak"],
                "unit": dom["unit"], "frac": dom["frac"], "traffic": dom_traffic,
                "traffic_unit": "bytes per launch (HBM read + write)",
                "kernel": dom["name"], "ms_per_launch": dom["ms"],
                "work_per_launch": dom["work_per_launch"]}
    g_ms = sum(e["ms"] for e in stage_rows if e["bound"] == "hbm" and e["name"] != "head")
    g_bytes = sum(e["work_per_launch"] for e in stage_rows if e["bound"] == "hbm" and e["name"] != "head")
    m_ms = sum(e["ms"] for e in stage_rows if e["bound"] == "mfma")
    m_flops = sum(e["work_per_launch"] for e in stage_rows if e["bound"] == "mfma")

    p50 = p99 = g50 = g99 = None
    lat_stages = floor = None
    if not args.no_latency:
        lat_np = request_slice(batch, 0, cfg)
        lat_dev = binding.batch_to_device(lat_np, dev)
        lat_scores = torch.empty(lat_np["n_rows"], dtype=torch.float32, device=dev)
        p50, p99 = latency(model, lat_dev, lat_scores, args.latency_iters, torch, graph=False)
        binding.cold_profile_enable(model.h, True)
        for _ in range(20):
            model.score(lat_dev, scores=lat_scores)
        torch.cuda.synchronize()
        lst, lcalls = binding.cold_profile_read(model.h)
        binding.cold_profile_enable(model.h, False)
        lat_stages = {name: round(tot / max(lcalls, 1) * 1e3, 2) for name, tot in lst}
        log(f"2,000-ad request stages (us): {lat_stages}")
        try:
            g50, g99 = latency(model, lat_dev, lat_scores, args.latency_iters, torch, graph=True)
        except Exception as exc:  # graph capture is an optional measurement
            log(f"graph replay unavailable: {exc}")
        log(f"2,000-ad request latency p50 {p50:.4f} ms (graph {g50}), p99 {p99:.4f} ms")
        floor = launch_sync_floor(torch, dev, args.latency_iters)
        log(f"host floor: one trivial kernel launched and synchronised, p50 {floor:.4f} ms")

    if args.no_latency:
        args.batching, args.serving_streams, args.topn, args.groups_sweep = "", "", 0, ""
    batching = None
    if args.batching:
        sizes = [int(v) for v in args.batching.split(",") if v]
        batching = batching_curve(model, batch, cfg, sizes, args.serving_iters, torch, binding)

    serving = None
    if args.serving_streams:
        ks = [int(v) for v in args.serving_streams.split(",") if v]
        serving = serving_curve(model, batch, cfg, ks, args.serving_iters, torch, binding)

    sweep = None
    if args.groups_sweep:
        counts = [int(v) for v in args.groups_sweep.split(",") if v]
        sweep = groups_sweep(synth.config(args.workload, n_requests=32, cand_per_request=2000),
                             counts, max(5, args.steps // 2), 3, torch, binding, synth, dev)

    topn = None
    if args.topn > 0:
        # per-request top-n by eCPM = CTR * bid after scoring (Section 2)
        bids = torch.from_numpy(synth.make_bids(cfg, R)).to(dev)
        req_off_t = dev_batch["req_off"]
        binding.select_topn(scores, bids, req_off_t, args.topn)
        torch.cuda.synchronize()
        t_ev0, t_ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        reps = 20
        t_ev0.record(stream)
        for _ in range(reps):
            binding.select_topn(scores, bids, req_off_t, args.topn)
        t_ev1.record(stream)
        torch.cuda.synchronize()
        batch_us = t_ev0.elapsed_time(t_ev1) / reps * 1e3
        one_off = req_off_t[:2].clone()
        one_off[1] = min(cfg.cand_per_request, R)
        t_ev0.record(stream)
        for _ in range(reps):
            binding.select_topn(scores, bids, one_off, args.topn)
        t_ev1.record(stream)
        torch.cuda.synchronize()
        one_us = t_ev0.elapsed_time(t_ev1) / reps * 1e3
        topn = {"n": args.topn, "us_per_batch": round(batch_us, 2),
                "rows_per_s": round(R / (batch_us * 1e-6), 1),
                "us_one_request": round(one_us, 2),
                "share_of_step": round(batch_us * 1e-3 / ms_per_step, 4)}
        log(f"top-{args.topn} by eCPM: {batch_us:.2f} us per batch, {one_us:.2f} us for one "
            f"{cfg.cand_per_request}-ad request")

    if args.copy_probe_mb > 0:
        n = args.copy_probe_mb << 20
        src = torch.ones(n, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"copy probe: {args.copy_probe_mb} MiB device-to-device")
        del src, dst

    gref = None
    if not args.no_latency:
        gref = gather_reference(cfg, batch, tables, 20, torch, dev)
        if gref:
            gs = next((e for e in stage_rows if e["name"] == "gather_se"), None)
            if gs:
                gref["gather_se_us"] = round(gs["ms"] * 1e3, 2)
            log(f"plain gather of the same rows: {gref['probe_us']} us (probe), "
                f"{gref['vendor_index_select_us']} us (torch.index_select); "
                f"gather_se {gref.get('gather_se_us')} us")

    others = None
    names = [w for w in args.other_workloads.split(",") if w and w != cfg.name]
    if names and not args.no_latency:
        others = [time_workload(w, args.steps, args.warmup, torch, binding, synth, dev) for w in names]

    cpu = parity = cpu1 = None
    if not args.no_cpu_baseline:
        cpu, parity, cpu1 = cpu_baseline(cfg, batch, params, args.cpu_seconds,
                                         gpu_scores=scores.cpu().numpy(),
                                         one_core_s=args.cpu_one_core_seconds)
        log(f"cpu baseline {cpu}; one core {cpu1}")
        log(f"parity over the checked rows: {parity}")

    out = {
        "metric": "candidate ads scored/sec on 1 GPU; p50 latency of a 2,000-ad request",
        "value": round(value, 1), "unit": "ads/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 5),
        "ms_per_step_with_stage_events": round(ms_profiled, 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": cfg.dtype, "data": "synthetic",
        "config": {"workload": cfg.name, "requests": cfg.n_requests,
                   "candidates_per_request": cfg.cand_per_request, "rows": R,
                   "groups": cfg.n_groups, "emb_dim": cfg.emb_dim, "vocab": cfg.vocab,
                   "widths": list(cfg.widths), "parallelism": "none (1 GPU)",
                   "cross_features": "built on the GPU from user/ad id pairs" if cfg.cross_pairs
                   else "ids given per row", "se_form": cfg.se_form},
        "p50_latency_ms": None if p50 is None else round(p50, 4),
        "p99_latency_ms": None if p99 is None else round(p99, 4),
        "p50_latency_graph_ms": None if g50 is None else round(g50, 4),
        "launch_sync_floor_ms": None if floor is None else round(floor, 4),
        "latency_stages_us": lat_stages,
        "p99_latency_graph_ms": None if g99 is None else round(g99, 4),
        "roofline": roofline,
        "roofline_gather_se": {"bound": "hbm", "achieved": round(g_bytes / (g_ms * 1e-3) / 1e9, 1),
                               "peak": PEAK_HBM_GBS, "unit": "GB/s",
                               "frac": round(g_bytes / (g_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)},
        "roofline_mlp": {"bound": "mfma", "achieved": round(m_flops / (m_ms * 1e-3) / 1e12, 2),
                         "peak": PEAK_MFMA_TFLOPS[cfg.dtype], "unit": "TFLOP/s",
                         "frac": round(m_flops / (m_ms * 1e-3) / 1e12 / PEAK_MFMA_TFLOPS[cfg.dtype], 4)},
        "stages": [dict({k: e[k] for k in ("name", "ms", "bound", "achieved", "unit", "frac")},
                        traffic=(traffic["stages"].get(e["name"]) if traffic else None))
                   for e in stage_rows],
        "cpu_baseline": cpu,
        "cpu_baseline_one_core": cpu1,
        "parity": parity,
        "topn": topn,
        "groups_sweep": sweep,
        "serving_streams": serving,
        "serving_batching": batching,
        "other_workloads": others,
        "gather_reference": gref,
        "usable_requests_per_s": None if not batching else {
            f"p99<={lim}ms": max([e["requests_per_s"] for e in batching if e["p99_ms"] <= lim],
                                 default=None) for lim in (0.1, 0.5, 1.0)},
    }
    print(json.dumps(out), flush=True)
    model.close()


if __name__ == "__main__":
    main()
