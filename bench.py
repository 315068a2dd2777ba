#!/usr/bin/env python3
"""Benchmark: one decode step of ragged paged attention over a compressed KV cache.

Default workload: the Qwen2.5-32B-shaped multi-turn decode step (64 layers run
back to back, batch 64, 64 query / 8 KV heads, head_dim 128, bf16, lognormal
contexts with median 16384, 20 % of (layer, head) pairs retaining 60-100 % and
the rest 3-15 %, page size 16, groups of 2 heads).  A step is the 64 per-layer
tg_decode calls (split-KV attention + log-sum-exp merge) with every input
already resident in HBM; host planning is done before the timed region and
reported separately as plan_build_us.

Prints ONE JSON line.  `value` is KV GB/s: the algorithmic retained-KV bytes
of a step (sum over requests, layers and KV heads of kv_len * 2 * d * 2 bytes)
divided by the measured step time.

    python bench.py [--steps K] [--warmup W] [--config 3] [--mode aot|naive|uniform]
    python bench.py --config 5             # chunked prefill + compression of the chunk
    python bench.py --compress-chunk C     # chunk compression alone, chunk of C tokens
    python bench.py --memory               # host only: memory reclaimed per paging scheme
    python bench.py --plan-reuse           # planning cost vs decode step, 28 to 80 layers
    python bench.py --tail-analysis        # decode layer tail: per-worker speed, per-XCD speed, weights
    python bench.py --lifecycle            # host only: calibration, reservation threads, release
    python bench.py --copy-probe BYTES     # plain copy kernel, for counter calibration
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
HBM_PEAK_GBS = 8000.0
METRIC = "ragged paged decode attn: KV GB/s, % of HBM peak, µs/decode step"
DECODE_SRC = os.path.join(ROOT, "paper_2606_06302_amd", "csrc", "tg_decode.hip")
PREFILL_SRC = os.path.join(ROOT, "paper_2606_06302_amd", "csrc", "tg_prefill.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "decode_traffic.json")
PREFILL_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "prefill_traffic.json")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def source_sha(src=DECODE_SRC):
    h = hashlib.sha256()
    for p in (src, os.path.join(ROOT, "paper_2606_06302_amd", "csrc", "tg_device.h")):
        h.update(open(p, "rb").read())
    return h.hexdigest()[:16]


def copy_probe(nbytes):
    import torch
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": nbytes}))


def host_cores():
    """The host's CPU share for the oracle runs: OMP_NUM_THREADS when the environment sets it."""
    return min(len(os.sched_getaffinity(0)), int(os.environ.get("OMP_NUM_THREADS", "0")) or 10**6)


def compress_kernel_name(chunk_len):
    from paper_2606_06302_amd import tangram as tg
    if chunk_len <= tg.TG_COMPRESS_ONE_LAUNCH_MAX_CHUNK:
        return "tg_compress (one launch: each item's wave selects its unit from registers and copies its ranks)"
    return "tg_compress (select + copy launches)"


def measured_traffic(workload, mode=None, n_bins=None, path=TRAFFIC_FILE, src=DECODE_SRC):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they were
    taken on the current kernel source and the same workload (and plan); else None."""
    try:
        rec = json.load(open(path))
    except (OSError, ValueError):
        return None
    if (rec.get("source_sha") != source_sha(src) or rec.get("workload") != workload or rec.get("mode") != mode
            or rec.get("n_bins") != n_bins):
        return None
    return rec.get("hbm_bytes_per_launch")


def cpu_baseline(session, seconds, threads=1, seed=7):
    """The fp64 oracle on a bounded sample of the same workload, timed on the host with BLAS
    limited to `threads` threads."""
    sys.path.insert(0, ROOT)
    from threadpoolctl import threadpool_limits

    import oracle
    import torch
    wl, t = session.wl, session.t
    g = wl.geom
    rng = np.random.default_rng(seed)
    order = [(int(b), int(l)) for b, l in zip(rng.integers(0, wl.batch, 10**4), rng.choice(session.layers, 10**4))]
    done_bytes, spent, pairs, max_abs = 0, 0.0, 0, 0.0
    P, G, L = g.page_size, g.num_groups, g.num_layers
    with threadpool_limits(limits=threads):
        for b, l in order:
            if spent >= seconds:
                break
            heads = [(b, h) for h in range(g.num_kv_heads)]
            # copy this request's pages of layer l back to the host (not timed)
            need = []
            for _, h in heads:
                base = int(t.pt_offsets[(b * L + l) * G + t.group_of[l, h]])
                need.append(t.pt_pages[base: base + (int(t.kv_len[b, l, h]) + P - 1) // P])
            idx = np.unique(np.concatenate(need)).astype(np.int64)
            sub = session.pool[torch.from_numpy(idx).cuda()].float().cpu().numpy().astype(np.float64)
            remap = np.full(t.pool_pages, -1, dtype=np.int64)
            remap[idx] = np.arange(len(idx))
            q = session.q[l].float().cpu().numpy().astype(np.float64)
            t0 = time.perf_counter()
            O, _ = oracle.decode_attention(q, sub, l, geom=g, batch=wl.batch, kv_len=t.kv_len, offsets=t.pt_offsets,
                                           pages=remap[t.pt_pages], group_of=t.group_of, slot_of=t.slot_of,
                                           heads=heads)
            spent += time.perf_counter() - t0
            done_bytes += int(t.kv_len[b, l].sum()) * 2 * g.head_dim * (2 if wl.dtype == "bf16" else 4)
            pairs += 1
            got = session.out[l, b].float().cpu().numpy().astype(np.float64)
            max_abs = max(max_abs, float(np.abs(got - O[b]).max()))
    return {"value": done_bytes / spent / 1e9, "unit": "GB/s", "cores": threads, "kind": "oracle",
            "sample": f"{pairs} (request, layer) pairs x all {g.num_kv_heads} KV heads of the same workload, "
                      f"{done_bytes / 1e9:.3f} GB of retained KV, {spent:.1f} s, BLAS limited to {threads} "
                      f"thread{'s' if threads > 1 else ''}",
            "gpu_vs_oracle_max_abs": max_abs}


MFMA_BF16_PEAK_TFLOPS = 2500.0
MALL_FLUSH_BYTES = 512 << 20


def step_stats(run, stream, n, flush):
    """Per-step times (ms) of n steps, HIP events on the launch stream around each; with `flush`, a 512 MB
    read on the same stream before every step evicts the 256 MB MALL, so no step reads a previous step's
    data from it (a read, not a write: dirty lines left by a write would be written back during the next
    step and charged to it).  Returns (median, p10, p90)."""
    import torch
    buf = torch.ones(MALL_FLUSH_BYTES // 4, dtype=torch.int32, device="cuda") if flush else None
    evs = []
    with torch.cuda.stream(stream):
        for _ in range(n):
            if buf is not None:
                buf.max()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            run()
            b.record(stream)
            evs.append((a, b))
    torch.cuda.synchronize()
    t = np.array([a.elapsed_time(b) for a, b in evs])
    return float(np.median(t)), float(np.percentile(t, 10)), float(np.percentile(t, 90))


def prefill_cpu_baseline(ps, seconds, seed=9, threads=1):
    """The fp64 oracle's chunked-prefill attention on sampled (request, query head) rows of the same
    workload, timed on the host with `threads` BLAS threads; TFLOP/s of those rows' algorithmic flops."""
    sys.path.insert(0, ROOT)
    from threadpoolctl import threadpool_limits

    import oracle
    import torch
    wl, t, g = ps.wl, ps.t, ps.wl.geom
    C, P, G, L = wl.chunk_len, g.page_size, g.num_groups, g.num_layers
    rng = np.random.default_rng(seed)
    f = lambda x: x.float().cpu().numpy().astype(np.float64)
    q, k, v = f(ps.q), f(ps.k_new), f(ps.v_new)
    got = f(ps.out)
    spent, flops, rows, max_abs = 0.0, 0, 0, 0.0
    with threadpool_limits(limits=threads):
        while spent < seconds and rows < 4096:
            b, qh = int(rng.integers(0, wl.batch)), int(rng.integers(0, g.num_q_heads))
            h = qh // g.gqa
            n = int(ps.hist[b, ps.layer, h])
            base = int(t.pt_offsets[(b * L + ps.layer) * G + t.group_of[ps.layer, h]])
            idx = t.pt_pages[base: base + (n + P - 1) // P].astype(np.int64)
            sub = ps.pool[torch.from_numpy(idx).cuda()].float().cpu().numpy().astype(np.float64)
            remap = np.full(t.pool_pages, -1, dtype=np.int64)
            remap[idx] = np.arange(len(idx))
            t0 = time.perf_counter()
            ref = oracle.prefill_attention(q, k, v, sub, ps.layer, geom=g, kv_len=ps.hist, offsets=t.pt_offsets,
                                           pages=remap[t.pt_pages], group_of=t.group_of, slot_of=t.slot_of,
                                           rows=[(b, qh)])
            spent += time.perf_counter() - t0
            flops += 4 * g.head_dim * (n * C + C * (C + 1) // 2)
            rows += 1
            max_abs = max(max_abs, float(np.abs(got[b, :, qh] - ref[b, :, qh]).max()))
    return {"value": flops / spent / 1e12, "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "sample": f"{rows} (request, query head) rows of the same chunk, all {C} query positions each, "
                      f"{flops / 1e9:.2f} GFLOP, {spent:.1f} s, BLAS limited to {threads} thread"
                      f"{'s' if threads > 1 else ''}",
            "gpu_vs_oracle_max_abs": max_abs}


def bench_prefill(args):
    """One layer of chunked prefill with its compression (bf16): ragged chunked-prefill attention
    (MFMA) over the compressed history, then the chunk's K/V compressed into the reserved pages."""
    import dataclasses

    import torch
    from paper_2606_06302_amd import tangram as tg
    from paper_2606_06302_amd.runner import CompressSession, PrefillSession, Tables
    from workloads import config
    wl5 = config(5)
    C, B = wl5.chunk_len, wl5.batch
    g = wl5.geom
    # the reservation covers each request's whole context: history plus this chunk
    wl = dataclasses.replace(wl5, ctx_len=wl5.ctx_len + C)
    log(f"[bench] workload {wl.name}: tables, pool, chunk inputs")
    tables = Tables(wl)
    starts, toks = wl5.ctx_len, np.full(B, C, dtype=np.int32)
    plan = tg.tg_compress_plan(g, B, 0, C, starts, toks, wl.ratio, wl.budget, tables.kv_len, tables.pt_offsets,
                               tables.group_of, tables.slot_of, 32)
    hist = plan["write_begin"].reshape(B, 1, g.num_kv_heads)     # ceil(r * 16384): Eq. 4 on the history
    s = PrefillSession(wl, tables=tables, hist_len=hist)
    cs = CompressSession(wl, tables, s.pool, starts, toks, k_new=s.k_new, v_new=s.v_new)
    torch.cuda.synchronize()
    flops = s.flops()
    comp_bytes = cs.traffic_bytes()
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        for _ in range(args.warmup):
            s.run(stream)
            cs.run(stream)
        stream.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(args.steps):
            s.run(stream)
            cs.run(stream)
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / args.steps
        # per-kernel times, events on the launch stream
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        pre_ms = comp_ms = 0.0
        nrep = max(1, min(args.steps, 10))
        for _ in range(nrep):
            ev[0].record(stream)
            s.run(stream)
            ev[1].record(stream)
            cs.run(stream)
            ev[2].record(stream)
            torch.cuda.synchronize()
            pre_ms += ev[0].elapsed_time(ev[1]) / nrep
            comp_ms += ev[1].elapsed_time(ev[2]) / nrep
    # timing protocol: per-step events after a MALL flush (the chunk's history fits the 256 MB MALL)
    med, p10, p90 = step_stats(lambda: (s.run(stream), cs.run(stream)), stream, max(args.steps, 50), True)
    tflops = flops / (med * 1e-3) / 1e12
    pre_tflops = flops / (pre_ms * 1e-3) / 1e12
    comp_gbs = comp_bytes / (comp_ms * 1e-3) / 1e9
    res = {
        "metric": "ragged chunked prefill attn: TFLOP/s (bf16 MFMA)", "value": round(tflops, 2), "unit": "TFLOP/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "timing": "value from the median of per-step HIP events, each step after a 512 MB MALL-evicting read; "
                  "ms_per_step is the plain average of the K back-to-back steps",
        "step_ms_median": round(med, 4), "step_ms_p10": round(p10, 4), "step_ms_p90": round(p90, 4),
        "config": {"workload": wl.name, "batch": B, "chunk_len": C, "q_heads": g.num_q_heads,
                   "kv_heads": g.num_kv_heads, "head_dim": g.head_dim, "history_ctx": int(wl5.ctx_len[0]),
                   "flops_per_step": flops, "step": "chunk attention over the compressed history, then the "
                   "chunk's K/V compressed into the reserved pages", "parallelism": "single GPU"},
        "roofline": {"bound": "mfma", "achieved": round(pre_tflops, 2), "peak": MFMA_BF16_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(pre_tflops / MFMA_BF16_PEAK_TFLOPS, 4),
                     "traffic": measured_traffic(wl.name, path=PREFILL_TRAFFIC_FILE, src=PREFILL_SRC),
                     "min_hbm_bytes_per_launch": s.min_hbm_bytes(),
                     "kernel": "tg_prefill_kernel", "avg_launch_us": round(pre_ms * 1e3, 2),
                     "algorithmic_flops_per_launch": flops},
        "compress": {"bound": "hbm", "achieved": round(comp_gbs, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(comp_gbs / HBM_PEAK_GBS, 4), "kernel": compress_kernel_name(C),
                     "avg_launch_us": round(comp_ms * 1e3, 2), "algorithmic_bytes_per_launch": comp_bytes,
                     "kept_rows": int(cs.plan["keep_count"].sum()), "work_items": cs.plan["num_items"]},
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline:
        log(f"[bench] cpu_baseline: oracle on sampled rows (~{args.cpu_seconds:.0f} s)")
        res["cpu_baseline"] = prefill_cpu_baseline(s, args.cpu_seconds)
        cores = host_cores()
        if cores > 1:
            res["cpu_baseline_all_cores"] = prefill_cpu_baseline(s, args.cpu_seconds * 2 / 3, seed=11, threads=cores)
    print(json.dumps(res), flush=True)


def bench_compress(args):
    """Compression of one prefill chunk into the ragged cache, alone: config 5's requests and ratios
    with a chunk of args.compress_chunk tokens after the 16384-token history."""
    import dataclasses

    import torch
    from paper_2606_06302_amd.runner import CompressSession, Tables
    from workloads import S_POOL, config, device_normal_, page_elems
    wl5 = config(5)
    C, B = args.compress_chunk, wl5.batch
    wl = dataclasses.replace(wl5, ctx_len=wl5.ctx_len + C, chunk_len=C)
    g = wl.geom
    log(f"[bench] chunk compression, {B} requests x {g.num_kv_heads} KV heads, chunk {C}")
    t = Tables(wl)
    pool = torch.empty(t.pool_pages * page_elems(g), dtype=torch.bfloat16, device="cuda")
    device_normal_(pool, wl, S_POOL, wl.kv_scale)
    pool = pool.view(t.pool_pages, 2, g.heads_per_group, g.page_size, g.head_dim)
    cs = CompressSession(wl, t, pool, wl5.ctx_len, np.full(B, C, dtype=np.int32),
                         rows_per_item=args.rows_per_item or 32)
    nbytes = cs.traffic_bytes()
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        for _ in range(args.warmup):
            cs.run(stream)
        stream.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(args.steps):
            cs.run(stream)
        e1.record(stream)
        torch.cuda.synchronize()
    us = e0.elapsed_time(e1) / args.steps * 1e3
    gbs = nbytes / (us * 1e-6) / 1e9
    res = {"metric": "chunk compression into ragged pages: GB/s of algorithmic HBM traffic", "value": round(gbs, 2),
           "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
           "ms_per_step": round(us / 1e3, 5), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
           "dtype": "bf16", "data": "synthetic",
           "config": {"workload": f"chunk-compression-bf16-c{C}", "batch": B, "chunk_len": C,
                      "kv_heads": g.num_kv_heads, "head_dim": g.head_dim, "history_ctx": int(wl5.ctx_len[0]),
                      "rows_per_item": args.rows_per_item or 32, "kept_rows": int(cs.plan["keep_count"].sum()),
                      "work_items": cs.plan["num_items"], "parallelism": "single GPU"},
           "roofline": {"bound": "hbm", "achieved": round(gbs, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                        "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": None,
                        "kernel": compress_kernel_name(C), "avg_launch_us": round(us, 2),
                        "algorithmic_bytes_per_launch": nbytes},
           "cpu_baseline": None}
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = compress_cpu_baseline(cs, args.cpu_seconds)
    print(json.dumps(res), flush=True)


def compress_cpu_baseline(cs, seconds, seed=10):
    """The oracle's compress_chunk on whole sampled requests of the same chunk (host, one thread);
    GB/s of the same algorithmic traffic."""
    sys.path.insert(0, ROOT)
    import oracle
    import torch
    wl, t, g = cs.wl, cs.t, cs.wl.geom
    L, G, P, H = g.num_layers, g.num_groups, g.page_size, g.num_kv_heads
    f = lambda x: x.float().cpu().numpy().astype(np.float64)
    k, v, sc = f(cs.k_new), f(cs.v_new), cs.scores.cpu().numpy()
    rng = np.random.default_rng(seed)
    spent, done, reqs, ok = 0.0, 0, 0, True
    sel = cs.wl.ratio
    while spent < seconds and reqs < wl.batch:
        b = int(rng.integers(0, wl.batch))
        lo, hi = b * L * G, (b + 1) * L * G
        idx = np.unique(t.pt_pages[t.pt_offsets[lo]: t.pt_offsets[hi]]).astype(np.int64)
        sub = cs.pool[torch.from_numpy(idx).cuda()].float().cpu().numpy().astype(np.float64)
        remap = np.full(t.pool_pages, -1, dtype=np.int64)
        remap[idx] = np.arange(len(idx))
        t0 = time.perf_counter()
        out, kept, cur, cnt = oracle.compress_chunk(k[b:b + 1], v[b:b + 1], sc[b:b + 1], sub, 0, geom=g,
                                                    ratio=sel[b:b + 1], capacity=t.kv_len[b:b + 1],
                                                    chunk_start=cs.chunk_start[b:b + 1],
                                                    chunk_tokens=cs.chunk_tokens[b:b + 1],
                                                    offsets=t.pt_offsets[lo: hi + 1], pages=remap[t.pt_pages],
                                                    group_of=t.group_of, slot_of=t.slot_of)
        spent += time.perf_counter() - t0
        ok &= bool(np.array_equal(out, sub))   # the GPU already wrote these rows: nothing may change
        n = int(cnt.sum())
        done += n * 2 * g.head_dim * 2 * 2 + int(cs.chunk_tokens[b]) * H * 4 + n * 8
        reqs += 1
    return {"value": done / spent / 1e9, "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"{reqs} whole requests (all {H} KV heads) of the same chunk, {spent:.1f} s",
            "gpu_matches_oracle": ok}


def bench_tail(args):
    """Where the decode layer's tail comes from (sequential-fill plan, HIP-graph step): per-worker
    stamps give every worker's pages per microsecond; their repeatability between two stamped runs,
    their spread over the 8 XCDs, and the step time after re-planning with per-bin or per-XCD bin
    weights taken from one stamped step."""
    import torch
    sys.path.insert(0, ROOT)
    from paper_2606_06302_amd import tangram as tg
    from paper_2606_06302_amd.runner import REALTIME_HZ, DecodeSession
    from workloads import config
    wl = config(args.config)
    s = DecodeSession(wl, mode=tg.TG_PLAN_AOT_FILL, fill="device")
    stream = torch.cuda.Stream()
    kv = s.t.kv_bytes()
    us = 1e6 / REALTIME_HZ

    def step_gbs(n=30):
        with torch.cuda.stream(stream):
            graph = s.capture_step(stream)
            for _ in range(3):
                graph.replay()
            stream.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(n):
                graph.replay()
            e1.record(stream)
            stream.synchronize()
        return kv / (e0.elapsed_time(e1) / n * 1e-3) / 1e9

    def stamped():
        """per layer: relative speed per bin (NaN for empty bins), span and mean busy time (us)"""
        speed, span, busy = {}, [], []
        for l in s.layers:
            t = s.stamp_layer(l, stream)
            pages = s.bin_pages(l)
            b = np.maximum(t[:, 1] - t[:, 0], 1)
            sp = np.where(pages > 0, pages / b, np.nan)
            speed[l] = sp / np.nanmean(sp)
            span.append((t[:, 1].max() - t[:, 0].min()) * us)
            busy.append(b[pages > 0].mean() * us)
        return speed, float(np.mean(span)), float(np.mean(busy))

    def row(name):
        gbs = step_gbs()
        sp, span, busy = stamped()
        log(f"[bench] {name}: {gbs:.1f} GB/s; mean layer span {span:.1f} us, mean worker busy {busy:.1f} us")
        return {"plan": name, "GBps": round(gbs, 1), "layer_span_us": round(span, 1),
                "worker_busy_us": round(busy, 1), "busy_over_span": round(busy / span, 4)}, sp

    step_gbs(5)
    rows = []
    r, sp0 = row("equal bins")
    rows.append(r)
    sp1, _, _ = stamped()
    xcd = (np.arange(s.n_bins) // s.workers_per_wg()) % 8
    corr = [np.corrcoef(sp0[l][np.isfinite(sp0[l])], sp1[l][np.isfinite(sp1[l])])[0, 1] for l in s.layers]
    per_xcd = np.array([[np.nanmean(sp0[l][xcd == k]) for k in range(8)] for l in s.layers])
    cv = [np.nanstd(sp0[l]) for l in s.layers]
    within = [np.nanstd(sp0[l] / per_xcd[i][xcd]) for i, l in enumerate(s.layers)]
    s.set_bin_weights({l: np.maximum(1, np.round(1000 * np.nan_to_num(sp0[l], nan=1.0))).astype(np.int32)
                       for l in s.layers})
    r, _ = row("per-bin weights from one stamped step")
    rows.append(r)
    s.set_bin_weights({l: np.maximum(1, np.round(1000 * per_xcd[i][xcd] / per_xcd[i].mean())).astype(np.int32)
                       for i, l in enumerate(s.layers)})
    r, _ = row("per-layer per-XCD weights from one stamped step")
    rows.append(r)
    out = {"metric": "decode layer tail analysis (per-worker stamps)", "data": "synthetic",
           "config": {"workload": wl.name, "plan": "fill", "n_bins": s.n_bins, "launch": "hip graph"},
           "speed_cv_median": round(float(np.median(cv)), 4),
           "speed_cv_within_xcd_median": round(float(np.median(within)), 4),
           "speed_corr_between_runs_median": round(float(np.median(corr)), 3),
           "per_xcd_speed_mean": [round(float(v), 3) for v in per_xcd.mean(0) / per_xcd.mean()],
           "per_xcd_speed_min": [round(float(v), 3) for v in (per_xcd / per_xcd.mean(1, keepdims=True)).min(0)],
           "per_xcd_speed_max": [round(float(v), 3) for v in (per_xcd / per_xcd.mean(1, keepdims=True)).max(0)],
           "rows": rows}
    print(json.dumps(out), flush=True)


def bench_memory(args):
    """Memory reclaimed by ragged paging (host, integer; no GPU): KV slots each scheme allocates for the
    same retained lengths, per heads-per-group and grouping, and the block-table build time."""
    sys.path.insert(0, ROOT)
    from paper_2606_06302_amd import tangram as tg
    from workloads import Geometry, config
    rows = []
    for cfg in (2, 3, 4, 5):
        wl = config(cfg)
        g = wl.geom
        esz = 4 if wl.dtype == "f32" else 2
        for Hp in (1, 2, 4, 8):
            geom = Geometry(g.num_layers, g.num_kv_heads, g.num_q_heads, g.head_dim, g.page_size, Hp)
            for grouping, gname in ((tg.TG_GROUP_CLUSTERED, "clustered"), (tg.TG_GROUP_ADJACENT, "adjacent")):
                _, gof, _ = tg.tg_cluster_heads(geom, wl.budget, grouping)
                f = tg.tg_memory_footprint(geom, wl.ctx_len, wl.ratio, None, gof)
                need = f["ragged_pages"]
                free = np.arange(need, dtype=np.int32)
                reps = 3
                tg.tg_reserve(geom, wl.ctx_len, wl.ratio, None, gof, free, need)   # untimed: first touch
                t0 = time.perf_counter()
                for _ in range(reps):
                    tg.tg_reserve(geom, wl.ctx_len, wl.ratio, None, gof, free, need)
                us = (time.perf_counter() - t0) / reps * 1e6
                full = f["full_slots"]
                rows.append({"workload": wl.name, "heads_per_group": Hp, "grouping": gname,
                             "full_GB": round(full * 2 * g.head_dim * esz / 1e9, 3),
                             "retained_frac": round(f["retained_slots"] / full, 4),
                             "monolithic_frac": round(f["monolithic_slots"] / full, 4),
                             "ragged_frac": round(f["ragged_slots"] / full, 4),
                             "reclaimed_vs_full": round(1 - f["ragged_slots"] / full, 4),
                             "reclaimed_monolithic": round(1 - f["monolithic_slots"] / full, 4),
                             "page_tables": f["page_tables"], "pages": need,
                             "reserve_us": round(us, 1)})
                log(f"[bench] {wl.name} H_p={Hp} {gname}: ragged {f['ragged_slots'] / full:.3f} of full, "
                    f"monolithic {f['monolithic_slots'] / full:.3f}, reserve {us:.0f} us")
    print(json.dumps({"metric": "KV slots allocated per paging scheme (fraction of the full cache)",
                      "data": "synthetic", "rows": rows}), flush=True)


def bench_plan_reuse(args):
    """Planning cost against the decode step (the analog of the paper's Table 1) for four model shapes.
    One decode step = for every layer, the new token's K/V appended and attention over the cache: step_ms
    with tg_append, tg_decode and its merge launch (three launches per layer), fused_append_step_ms with the
    append inside the decode launch (tg_decode's append_k / append_v), one_launch_step_ms with the append
    and the merge inside it (merge_counters too).  Each form runs the same steps from the same live lengths.
    The ahead-of-time open-ended plans are built once, before the first step, and serve every step; a
    planner run at every step would cost plan_build_ms (host) + plan_upload_ms."""
    import torch
    from paper_2606_06302_amd import tangram as tg
    from paper_2606_06302_amd.device import upload_plan
    from paper_2606_06302_amd.runner import DecodeSession, Tables
    from workloads import MODEL_SHAPES, model_step
    rows = []
    steps, warmup = args.steps, args.warmup
    for name in MODEL_SHAPES:
        wl = model_step(name)
        g = wl.geom
        log(f"[bench] {wl.name}: {g.num_layers} layers, tables and pool")
        t = Tables(wl, headroom=np.full(wl.batch, steps + warmup + 2, dtype=np.int32))
        s = DecodeSession(wl, tables=t, mode=tg.TG_PLAN_AOT_FILL, open_end=True)
        s.enable_append()
        torch.cuda.synchronize()
        # host planning of every layer, as a per-step planner would have to redo it
        t0 = time.perf_counter()
        plans = [tg.tg_build_plan(g, wl.batch, l, t.kv_len, t.pt_offsets, t.group_of, t.slot_of,
                                  tg.TG_PLAN_AOT_FILL | tg.TG_PLAN_OPEN_END, s.n_bins) for l in s.layers]
        plan_ms = (time.perf_counter() - t0) * 1e3
        t0 = time.perf_counter()
        for p_ in plans:
            upload_plan(g, wl.batch, p_, "cuda")
        torch.cuda.synchronize()
        upload_ms = (time.perf_counter() - t0) * 1e3
        stream = torch.cuda.Stream()

        live0 = s.live_len.clone()

        def timed_steps():
            s.live_len.copy_(live0)   # every form appends the same tokens at the same places
            with torch.cuda.stream(stream):
                for _ in range(warmup):
                    s.run_decode_step(stream)
                stream.synchronize()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                for _ in range(steps):
                    s.run_decode_step(stream)
                e1.record(stream)
                torch.cuda.synchronize()
            return e0.elapsed_time(e1) / steps

        step_ms = timed_steps()
        kv = int(s.live_len.sum().item()) * 2 * g.head_dim * 2
        s.enable_append(fused=True)
        fused_ms = timed_steps()
        counters = torch.zeros(wl.batch * g.num_kv_heads, dtype=torch.int32, device="cuda")
        for a in s.append_decode_args.values():
            a.merge_counters = counters.data_ptr()
        one_ms = timed_steps()
        assert int(s.full.item()) == 0, "decode headroom exhausted"
        rows.append({"model": name, "layers": g.num_layers, "q_heads": g.num_q_heads, "kv_heads": g.num_kv_heads,
                     "batch": wl.batch, "step_ms": round(step_ms, 3), "fused_append_step_ms": round(fused_ms, 3),
                     "one_launch_step_ms": round(one_ms, 3),
                     "kv_GB_per_step": round(kv / 1e9, 2),
                     "kv_GBps": round(kv / (step_ms * 1e-3) / 1e9, 1),
                     "plan_build_ms": round(plan_ms, 3), "plan_upload_ms": round(upload_ms, 3),
                     "replan_share": round((plan_ms + upload_ms) / (plan_ms + upload_ms + step_ms), 4),
                     "aot_plan_share": 0.0})
        log(f"[bench]   step {step_ms:.3f} ms ({rows[-1]['kv_GBps']} GB/s), append in decode {fused_ms:.3f} ms, "
            f"append and merge in decode {one_ms:.3f} ms, "
            f"plan {plan_ms:.2f} ms + upload "
            f"{upload_ms:.2f} ms")
        del s, t, plans
        torch.cuda.empty_cache()
    print(json.dumps({"metric": "planning cost vs decode step (append + attention, all layers)",
                      "data": "synthetic", "steps": steps, "warmup": warmup, "rows": rows}), flush=True)


def bench_lifecycle(args):
    """Host only: budget calibration from synthetic retention samples (B = min(1, mu + 2 sigma) over 50
    pilot samples, checked on 50 held-out ones), the reservation at one head per group with 1 and 16
    host threads, and releasing / readmitting a quarter of a batch."""
    sys.path.insert(0, ROOT)
    from paper_2606_06302_amd import tangram as tg
    from workloads import Geometry, config, retention_scores
    out = {"metric": "calibration and request lifecycle (host)", "data": "synthetic"}
    # calibration: a Llama-3.1-8B-shaped layer stack, 16384-token pilot contexts, rho = 0.3
    L, H, N, rho, alpha, n_pilot = 32, 8, 16384, 0.3, 2.0, 50
    t_ratio, pilot = 0.0, []
    for s_ in range(n_pilot):
        sc = retention_scores(77, s_, L, H, N)
        t0 = time.perf_counter()
        r, _ = tg.tg_implicit_ratios(sc, rho)
        t_ratio += time.perf_counter() - t0
        pilot.append(r)
    t0 = time.perf_counter()
    B = tg.tg_calibrate_budget(np.stack(pilot), alpha, 1.0 / N)
    t_cal = time.perf_counter() - t0
    over, excess, reserved = 0, [], []
    for s_ in range(n_pilot, 2 * n_pilot):
        r, _ = tg.tg_implicit_ratios(retention_scores(77, s_, L, H, N), rho)
        over += int((r > B).sum())
        excess.extend((r[r > B] - B[r > B]).tolist())
    for l in range(L):
        reserved.append(sum(math.ceil(float(B[l, h]) * N) for h in range(H)) / math.ceil(rho * H * N))
    out["calibration"] = {
        "layers": L, "kv_heads": H, "pilot_tokens": N, "rho": rho, "alpha": alpha, "pilot_samples": n_pilot,
        "implicit_ratio_ms_per_sample": round(t_ratio / n_pilot * 1e3, 2), "calibrate_ms": round(t_cal * 1e3, 3),
        "budget_mean": round(float(B.mean()), 4), "budget_min": round(float(B.min()), 4),
        "budget_max": round(float(B.max()), 4),
        "heldout_over_budget_frac": round(over / (n_pilot * L * H), 5),
        "heldout_mean_excess_ratio": round(float(np.mean(excess)) if excess else 0.0, 5),
        "reserved_over_global_budget": round(float(np.mean(reserved)), 4)}
    log(f"[bench] calibration: {out['calibration']}")
    # reservation at one head per group (32768 tables of the 64-layer decode workload)
    wl = config(3)
    g = wl.geom
    geom = Geometry(g.num_layers, g.num_kv_heads, g.num_q_heads, g.head_dim, g.page_size, 1)
    _, gof, _ = tg.tg_cluster_heads(geom, wl.budget)
    need = tg.tg_reserve(geom, wl.ctx_len, wl.ratio, None, gof, np.zeros(0, np.int32), 0,
                         size_query=True)["pages_needed"]
    free = np.random.default_rng(0).permutation(need).astype(np.int32)
    res_ms = {}
    for thr in (1, 16):
        os.environ["TG_HOST_THREADS"] = str(thr)
        best = []
        for _ in range(4):
            t0 = time.perf_counter()
            res = tg.tg_reserve(geom, wl.ctx_len, wl.ratio, None, gof, free, need)
            best.append(time.perf_counter() - t0)
        res_ms[thr] = round(min(best) * 1e3, 2)
    os.environ.pop("TG_HOST_THREADS", None)
    t0 = time.perf_counter()
    tg.tg_reserve(geom, wl.ctx_len, wl.ratio, None, gof, free, need, size_query=True)
    sq_ms = (time.perf_counter() - t0) * 1e3
    # a quarter of the batch finishes; the same number of requests is admitted from the freed pages
    fin = np.zeros(wl.batch, dtype=bool)
    fin[np.random.default_rng(1).permutation(wl.batch)[: wl.batch // 4]] = True
    t0 = time.perf_counter()
    freed, off, pages = tg.tg_release_requests(geom, res["pt_offsets"], res["pt_pages"], fin)
    t_rel = time.perf_counter() - t0
    t0 = time.perf_counter()
    again = tg.tg_reserve(geom, wl.ctx_len[fin], wl.ratio[fin], None, gof, freed, need)
    off2, pages2 = tg.tg_concat_tables(geom, off, pages, again["pt_offsets"], again["pt_pages"])
    t_adm = time.perf_counter() - t0
    out["reservation"] = {"workload": wl.name, "heads_per_group": 1, "tables": int(wl.batch * g.num_layers *
                          g.num_kv_heads), "pages": int(need), "size_query_ms": round(sq_ms, 3),
                          "reserve_ms_1_thread": res_ms[1], "reserve_ms_16_threads": res_ms[16],
                          "host_threads_available": os.cpu_count()}
    out["lifecycle"] = {"released_requests": int(fin.sum()), "released_pages": int(len(freed)),
                        "release_ms": round(t_rel * 1e3, 2), "readmit_and_concat_ms": round(t_adm * 1e3, 2),
                        "pages_conserved": bool(sorted(pages2.tolist()) == sorted(res["pt_pages"].tolist()))}
    log(f"[bench] reservation: {out['reservation']}")
    log(f"[bench] lifecycle: {out['lifecycle']}")
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", type=int, default=3)
    ap.add_argument("--mode", default="fill", choices=["aot", "fill", "naive", "uniform", "splitmap"])
    ap.add_argument("--n-bins", type=int, default=0)
    ap.add_argument("--split-target", type=int, default=0)
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--launch", default="auto", choices=["auto", "graph", "eager"],
                    help="how the timed steps are launched: a HIP graph replay or eager calls; auto = the graph for "
                         "multi-layer steps, eager calls for single-layer ones (each of those follows a MALL flush, "
                         "during which the host enqueues the step, and a graph replay adds dispatch latency)")
    ap.add_argument("--fused-merge", action="store_true",
                    help="merge split units inside the decode launch (merge_counters) instead of a second launch")
    ap.add_argument("--no-calibrate", action="store_true",
                    help="fill plans with equal bins (default: per-layer per-XCD bin weights from one stamped step)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--probe-workers", type=int, default=8192,
                    help="waves of the streaming-read ceiling probe (8 per SIMD by default)")
    ap.add_argument("--copy-probe", type=int, default=0)
    ap.add_argument("--compress-chunk", type=int, default=0,
                    help="time only the compression of a chunk of this many tokens (config 5's requests)")
    ap.add_argument("--rows-per-item", type=int, default=0)
    ap.add_argument("--tail-analysis", action="store_true",
                    help="per-worker stamps of the fill plan: speed spread, per-XCD speed, re-planning with weights")
    ap.add_argument("--plan-reuse", action="store_true",
                    help="planning cost against the decode step (append + attention) for 28 to 80 layers")
    ap.add_argument("--lifecycle", action="store_true",
                    help="host only: budget calibration, reservation threads, release and readmission")
    ap.add_argument("--memory", action="store_true",
                    help="host-only: memory reclaimed by ragged paging for each heads-per-group and grouping")
    ap.add_argument("--free-order", default="shuffled", choices=["shuffled", "sequential"],
                    help="order of the free page list (shuffled = seeded permutation of the pool)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: the library has no multi-GPU path (asked for --gpus {args.gpus}).",
              file=sys.stderr)
        sys.exit(2)
    if args.copy_probe:
        copy_probe(args.copy_probe)
        return
    if args.memory:
        return bench_memory(args)
    if args.lifecycle:
        return bench_lifecycle(args)

    import torch
    sys.path.insert(0, ROOT)
    from paper_2606_06302_amd import tangram as tg
    from paper_2606_06302_amd.runner import DecodeSession
    from workloads import config

    if args.compress_chunk:
        return bench_compress(args)
    if args.plan_reuse:
        return bench_plan_reuse(args)
    if args.tail_analysis:
        return bench_tail(args)
    if args.config == 5:
        return bench_prefill(args)
    mode = {"aot": tg.TG_PLAN_AOT, "fill": tg.TG_PLAN_AOT_FILL, "naive": tg.TG_PLAN_NAIVE,
            "uniform": tg.TG_PLAN_UNIFORM, "splitmap": tg.TG_PLAN_SPLIT_MAP}[args.mode]
    wl = config(args.config)
    log(f"[bench] workload {wl.name}: building tables, plans and a "
        f"{'device-filled' if args.config != 1 else 'host-filled'} pool")
    t0 = time.perf_counter()
    tables = None
    if args.free_order == "sequential":
        from paper_2606_06302_amd.runner import Tables
        t0_ = Tables(wl)
        tables = Tables(wl, free_pages=np.arange(t0_.pool_pages, dtype=np.int32), pool_pages=t0_.pool_pages)
    s = DecodeSession(wl, tables=tables, mode=mode, n_bins=args.n_bins or None,
                      split_target=args.split_target or None, fill="host" if args.config == 1 else "device",
                      fused_merge=args.fused_merge)
    torch.cuda.synchronize()
    log(f"[bench] setup {time.perf_counter() - t0:.1f} s: pool {s.t.pool_pages} pages "
        f"({s.pool.numel() * s.pool.element_size() / 1e9:.1f} GB), n_bins {s.n_bins}, "
        f"split_target {s.split_target}, plan build {s.plan_build_us / 1e3:.2f} ms")
    g = wl.geom
    kv_bytes_step = s.t.kv_bytes()
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        for _ in range(args.warmup):
            s.run_step(stream)
        stream.synchronize()
        xcd_speed = None
        if mode == tg.TG_PLAN_AOT_FILL and not args.no_calibrate:
            # ahead-of-time calibration (untimed, like the plan build): one stamped step measures
            # each XCD's pages per microsecond on every layer, and the layers' fill plans are
            # rebuilt with bin weights in proportion
            xcd_speed = s.calibrate_xcd_weights(stream, per_layer=True)
            log(f"[bench] per-XCD relative speed (mean over layers) "
                f"{np.round(xcd_speed.mean(0), 3).tolist()}; plans rebuilt")
            for _ in range(2):
                s.run_step(stream)
            stream.synchronize()
        log(f"[bench] warmup {args.warmup} steps done")
        # whole-step timing: the layers' launches captured once in a HIP graph, or eager calls
        use_graph = args.launch == "graph" or (args.launch == "auto" and g.num_layers > 1)
        graph = s.capture_step(stream) if use_graph else None
        if graph is not None:
            graph.replay()
            stream.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(args.steps):
            if graph is not None:
                graph.replay()
            else:
                s.run_step(stream)
        e1.record(stream)
        torch.cuda.synchronize()
        ms_per_step = e0.elapsed_time(e1) / args.steps
        log(f"[bench] timed {args.steps} steps: {ms_per_step:.3f} ms/step")
        # timing protocol: per-step distribution; single-layer workloads whose KV could sit in the 256 MB
        # MALL are flushed before every step (the 64-layer step streams ~85 GB and needs no flush)
        flush = g.num_layers == 1
        med, p10, p90 = step_stats((lambda: graph.replay()) if graph is not None else (lambda: s.run_step(stream)),
                                   stream, max(args.steps, 50), flush)
        # per-launch timing of the decode call (roofline), events on the launch stream
        nrep = max(1, min(args.steps, 5))
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in s.layers]
        lay_ms = np.zeros(len(s.layers))
        for _ in range(nrep):
            for i, l in enumerate(s.layers):
                evs[i][0].record(stream)
                s.run_layer(l, stream)
                evs[i][1].record(stream)
            torch.cuda.synchronize()
            lay_ms += np.array([a.elapsed_time(b) for a, b in evs])
        lay_ms /= nrep
        timeline = s.worker_timeline(stream)   # an extra untimed step with per-worker stamps
        busy = [(r["busy_max"], r["busy_mean"]) for r in timeline]
        # streaming-read ceiling of the same access pattern: the probe reads exactly the page slabs the
        # decode reads on a sample of layers, with the same number of workers and no arithmetic
        probe_layers = s.layers[:: max(1, len(s.layers) // 8)]
        t_probe = t_dec = 0.0
        probe_bytes = 0
        probe_workers = args.probe_workers
        out_ck = torch.zeros(probe_workers, dtype=torch.int32, device="cuda")
        for l in probe_layers:
            pages, slots = s.layer_slabs(l)
            dp, ds = torch.from_numpy(pages).cuda(), torch.from_numpy(slots).cuda()
            tg.tg_read_probe(g, s.tg_dtype, s.pool, dp, ds, probe_workers, out_ck, stream)   # untimed warm-up
            a_, b_, c_ = (torch.cuda.Event(enable_timing=True) for _ in range(3))
            a_.record(stream)
            tg.tg_read_probe(g, s.tg_dtype, s.pool, dp, ds, probe_workers, out_ck, stream)
            b_.record(stream)
            s.run_layer(l, stream)
            c_.record(stream)
            torch.cuda.synchronize()
            t_probe += a_.elapsed_time(b_)
            t_dec += b_.elapsed_time(c_)
            probe_bytes += len(pages) * 2 * g.page_size * g.head_dim * (2 if wl.dtype == "bf16" else 4)
    launch_bytes = np.array([s.t.kv_bytes(l) for l in s.layers], dtype=np.float64)
    achieved = float(launch_bytes.sum() / (lay_ms.sum() * 1e-3) / 1e9)
    imb = [s.bin_load_stats(l) for l in s.layers]
    planned_imbalance = float(np.mean([mx / mean for mx, mean in imb]))
    measured_imbalance = float(np.mean([mx / mean for mx, mean in busy]))
    value = kv_bytes_step / ((med if flush else ms_per_step) * 1e-3) / 1e9
    traffic = measured_traffic(wl.name, args.mode, s.n_bins)
    res = {
        "metric": METRIC, "value": round(value, 2), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": wl.dtype, "data": "synthetic",
        "timing": ("value from the median of per-step HIP events, each step after a 512 MB MALL-evicting read"
                   if flush else "value from K back-to-back steps between two synchronisations"),
        "step_ms_median": round(med, 4), "step_ms_p10": round(p10, 4), "step_ms_p90": round(p90, 4),
        "config": {"workload": wl.name, "layers": g.num_layers, "batch": wl.batch, "q_heads": g.num_q_heads,
                   "kv_heads": g.num_kv_heads, "head_dim": g.head_dim, "page_size": g.page_size,
                   "heads_per_group": g.heads_per_group, "plan": args.mode, "n_bins": s.n_bins,
                   "split_target": s.split_target, "kv_bytes_per_step": kv_bytes_step,
                   "free_order": args.free_order, "launch": "hip graph" if use_graph else "eager",
                   "merge": "in the decode launch" if args.fused_merge else "second launch",
                   "bin_weights": None if xcd_speed is None else "per-layer per-XCD speed from one stamped "
                                  "step (mean over layers " + str(np.round(xcd_speed.mean(0), 3).tolist()) + ")",
                   "parallelism": "single GPU"},
        "us_per_step": round((med if flush else ms_per_step) * 1e3, 1),
        "stream_ceiling": {"value": round(probe_bytes / (t_probe * 1e-3) / 1e9, 1), "unit": "GB/s",
                           "layers": len(probe_layers),
                           "workers": args.probe_workers,
                           "what": "tg_read_probe: the same page slabs as the decode, no arithmetic"},
        "frac_of_stream_ceiling": round(t_probe / t_dec, 4),
        "hbm_frac": round(value / HBM_PEAK_GBS, 4),
        "plan_build_us": round(s.plan_build_us, 1),
        "load_imbalance_planned": round(planned_imbalance, 4),
        "load_imbalance_measured": round(measured_imbalance, 4),
        "worker_timeline_us": {k: round(float(np.median([r[k] for r in timeline])), 2)
                               for k in ("span", "ramp", "tail", "busy_max", "busy_mean")},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": traffic,
                     "kernel": "tg_decode (split-KV decode + merge) per layer",
                     "avg_launch_us": round(float(lay_ms.mean()) * 1e3, 2),
                     "algorithmic_bytes_per_launch": round(float(launch_bytes.mean()))},
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline:
        log(f"[bench] cpu_baseline: oracle on a bounded sample (~{args.cpu_seconds:.0f} s)")
        res["cpu_baseline"] = cpu_baseline(s, args.cpu_seconds, threads=1)
        cores = host_cores()
        if cores > 1:
            res["cpu_baseline_all_cores"] = cpu_baseline(s, args.cpu_seconds * 2 / 3, threads=cores, seed=8)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
