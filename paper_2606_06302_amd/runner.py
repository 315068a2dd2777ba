"""Sets up one synthetic decode / prefill workload on the GPU and runs it through the C ABI.

Plumbing only: the host tables come from libtangram's tg_cluster_heads /
tg_reserve / tg_build_plan, device memory comes from torch, and every step of
the attention runs in libtangram's HIP kernels.
"""
from __future__ import annotations

import time

import numpy as np
import torch

from . import tangram as tg
from .device import bind_decode, to_device, upload_plan

TORCH_DTYPE = {"f32": torch.float32, "bf16": torch.bfloat16}
TG_DTYPE = {"f32": tg.TG_F32, "bf16": tg.TG_BF16}


class Tables:
    """Clustering + reservation of one workload (host arrays and device copies)."""

    def __init__(self, wl, free_pages=None, pool_pages=None, grouping=tg.TG_GROUP_CLUSTERED, device="cuda",
                 headroom=None):
        from workloads import free_list, pool_pages_for   # seeded inputs only
        g = wl.geom
        self.wl = wl
        self.perm, self.group_of, self.slot_of = tg.tg_cluster_heads(g, wl.budget, grouping)
        self.headroom = headroom
        if free_pages is None:
            need = tg.tg_reserve(g, wl.ctx_len, wl.ratio, None, self.group_of, np.zeros(0, np.int32), 0,
                                 size_query=True, headroom=headroom)["pages_needed"]
            pool_pages = pool_pages_for(need)
            free_pages = free_list(wl, pool_pages)
        self.pool_pages = int(pool_pages)
        self.free_pages = np.asarray(free_pages, dtype=np.int32)
        t0 = time.perf_counter()
        res = tg.tg_reserve(g, wl.ctx_len, wl.ratio, None, self.group_of, self.free_pages, self.pool_pages,
                            headroom=headroom)
        self.reserve_us = (time.perf_counter() - t0) * 1e6
        self.kv_len = res["kv_len"]
        self.group_len = res["group_len"]
        self.pt_offsets = res["pt_offsets"]
        self.pt_pages = res["pt_pages"]
        self.pages_needed = res["pages_needed"]
        self.device = device
        self.d_pt_pages = to_device(self.pt_pages if len(self.pt_pages) else np.zeros(1, np.int32), device)

    def kv_bytes(self, layer=None) -> int:
        """Algorithmic bytes of retained K and V (what the method must read)."""
        g = self.wl.geom
        esz = 4 if self.wl.dtype == "f32" else 2
        kv = self.kv_len if layer is None else self.kv_len[:, layer]
        return int(kv.sum()) * 2 * g.head_dim * esz


class DecodeSession:
    """Pool, queries, outputs and per-layer plans of one decode workload."""

    def __init__(self, wl, tables: Tables = None, mode=tg.TG_PLAN_AOT, n_bins=None, split_target=None,
                 fill="device", pool=None, q=None, want_lse=True, device="cuda", layers=None, open_end=False,
                 fused_merge=False):
        from workloads import S_POOL, S_Q, device_normal_, host_pool, host_q_decode, page_elems
        g = wl.geom
        self.wl, self.device = wl, device
        self.t = tables if tables is not None else Tables(wl, device=device)
        self.dtype = TORCH_DTYPE[wl.dtype]
        self.tg_dtype = TG_DTYPE[wl.dtype]
        if n_bins is None:
            n_bins = tg.tg_decode_max_ctas(g, self.tg_dtype, torch.device(device).index or 0)
        if split_target is None:
            split_target = 2 * n_bins   # measured best on the 64-layer step (bins x {1,2,4,8})
        self.mode, self.n_bins, self.split_target = mode, n_bins, split_target
        # open-ended plans: every unit's last chunk runs to the live length, so that the
        # plans built here serve every later decode step (tokens appended with append_layer)
        self.open_end = open_end
        self.live_len = to_device(self.t.kv_len, device) if open_end else None
        self.bin_weights = None
        L, B = g.num_layers, wl.batch
        self.layers = list(range(L)) if layers is None else list(layers)
        self._build_plans()
        # pool
        if pool is not None:
            self.pool = pool
        elif fill == "host":
            host = host_pool(wl, self.t.pool_pages)
            self.pool = torch.from_numpy(host).to(self.dtype).to(device)
        else:
            self.pool = torch.empty(self.t.pool_pages * page_elems(g), dtype=self.dtype, device=device)
            device_normal_(self.pool, wl, S_POOL, wl.kv_scale)
        self.pool = self.pool.view(self.t.pool_pages, 2, g.heads_per_group, g.page_size, g.head_dim)
        if q is not None:
            self.q = q
        elif fill == "host":
            self.q = torch.from_numpy(host_q_decode(wl)).to(self.dtype).to(device)
        else:
            self.q = torch.empty(L, B, g.num_q_heads, g.head_dim, dtype=self.dtype, device=device)
            device_normal_(self.q, wl, S_Q, wl.q_scale)
        self.out = torch.zeros(L, B, g.num_q_heads, g.head_dim, dtype=self.dtype, device=device)
        # arrival counters of the in-launch merge (zero; every call leaves them zero), shared by the layers'
        # calls, which run one after the other on a stream; None: the merge is a second launch
        self.merge_counters = (torch.zeros(B * g.num_kv_heads, dtype=torch.int32, device=device)
                               if fused_merge else None)
        self.lse = torch.zeros(L, B, g.num_q_heads, dtype=torch.float32, device=device) if want_lse else None
        self._bind()

    def _build_plans(self):
        g, B = self.wl.geom, self.wl.batch
        # timed: this is the host planning cost the paper's Table 1 measures for a runtime planner
        t0 = time.perf_counter()
        mode = self.mode | (tg.TG_PLAN_OPEN_END if self.open_end else 0)
        if self.mode == tg.TG_PLAN_SPLIT_MAP:
            # Algorithm 1 on the static budgets with N_CTA = n_bins: one row of S per layer
            S = tg.tg_split_map(g, self.wl.budget, self.t.perm, self.n_bins)
            weights = {l: S[l] for l in self.layers}
        elif isinstance(self.bin_weights, dict):
            weights = self.bin_weights
        else:
            weights = {l: self.bin_weights for l in self.layers}
        self.plans = {l: tg.tg_build_plan(g, B, l, self.t.kv_len, self.t.pt_offsets, self.t.group_of,
                                          self.t.slot_of, mode, self.n_bins, self.split_target,
                                          bin_weights=weights[l]) for l in self.layers}
        self.plan_build_us = (time.perf_counter() - t0) * 1e6
        self.dplans = {l: upload_plan(g, B, p, self.device) for l, p in self.plans.items()}

    def _bind(self):
        g, B = self.wl.geom, self.wl.batch
        for l in self.layers:
            bind_decode(self.dplans[l], g, B, self.tg_dtype, self.q[l], self.pool, self.t.d_pt_pages, self.out[l],
                        None if self.lse is None else self.lse[l], live_len=self.live_len, layer=l,
                        merge_counters=self.merge_counters)

    def item_tokens(self, l):
        """Tokens of every item of layer l's plan; open-ended items count up to the lengths the
        plan was built for."""
        items = self.plans[l]["items"]
        end = items["tok_end"].astype(np.int64)
        open_ = end < 0
        end[open_] = self.t.kv_len[items["b"][open_], l, items["kv_head"][open_]]
        return end - items["tok_begin"]

    def workers_per_wg(self):
        """Bins (workers) per workgroup of the decode kernel the library picks for this session:
        four waves, each its own worker, in the bf16 head-dim-128 kernel; one otherwise."""
        g = self.wl.geom
        return 4 if (self.tg_dtype == tg.TG_BF16 and g.head_dim == 128) else 1

    def calibrate_xcd_weights(self, stream=None, classes=8, per_layer=False):
        """Measures every worker's pages per microsecond over one stamped step and rebuilds the
        sequential-fill plans with bin weights in proportion to the speed of the worker's class.
        Worker k runs in workgroup k // w (w = workers_per_wg(): 4 for the bf16 head-dim-128 kernel,
        else 1); workgroups are dispatched round-robin over the `classes` XCDs, so class =
        (k // w) % classes.  With per_layer, each layer gets the speeds
        its own stamps show (the pattern differs from layer to layer); else one set pooled over the
        layers.  Returns the relative speeds: [classes], or [layers][classes] with per_layer."""
        assert self.mode == tg.TG_PLAN_AOT_FILL, "bin weights apply to the sequential-fill plan"
        pages = np.zeros((len(self.layers), classes))
        busy = np.zeros((len(self.layers), classes))
        for i, l in enumerate(self.layers):
            t = self.stamp_layer(l, stream)
            per_bin = self.bin_pages(l)
            cls = (np.arange(len(per_bin)) // self.workers_per_wg()) % classes
            np.add.at(pages[i], cls, per_bin)
            np.add.at(busy[i], cls, t[:, 1] - t[:, 0])

        def relative(p, b):
            sp = np.where(b > 0, p / np.maximum(b, 1), np.nan)
            sp = sp / np.nanmean(sp) if np.isfinite(sp).any() else np.ones_like(sp)
            return np.nan_to_num(sp, nan=1.0)

        cls = (np.arange(self.n_bins) // self.workers_per_wg()) % classes
        if per_layer:
            speed = np.stack([relative(pages[i], busy[i]) for i in range(len(self.layers))])
            self.set_bin_weights({l: np.maximum(1, np.round(1000 * speed[i][cls])).astype(np.int32)
                                  for i, l in enumerate(self.layers)})
        else:
            speed = relative(pages.sum(0), busy.sum(0))
            self.set_bin_weights(np.maximum(1, np.round(1000 * speed[cls])).astype(np.int32))
        return speed

    def enable_append(self, k_tok=None, v_tok=None, fused=False):
        """Device buffers for one decode step's new token per layer ([L][B][H][d] K and V) and the
        tg_append arguments of every layer; run_decode_step then appends before attending, with
        tg_append (two launches per layer) or, when fused, inside the decode launch (tg_decode's
        append_k / append_v: one launch per layer, the same results bit for bit)."""
        assert self.open_end, "appending needs open-ended plans and live lengths"
        g, B, dev = self.wl.geom, self.wl.batch, self.device
        shape = (g.num_layers, B, g.num_kv_heads, g.head_dim)
        self.k_tok = k_tok if k_tok is not None else torch.zeros(shape, dtype=self.dtype, device=dev)
        self.v_tok = v_tok if v_tok is not None else torch.zeros(shape, dtype=self.dtype, device=dev)
        self.full = torch.zeros(1, dtype=torch.int32, device=dev)
        self.d_offsets = to_device(self.t.pt_offsets, dev)
        self.d_group_of = to_device(self.t.group_of, dev)
        self.d_slot_of = to_device(self.t.slot_of, dev)
        self.append_args = {l: tg.make_append_args(g, B, l, self.tg_dtype, self.k_tok[l], self.v_tok[l], self.pool,
                                                   self.t.d_pt_pages, self.d_offsets, self.d_group_of,
                                                   self.d_slot_of, self.live_len, self.full) for l in self.layers}
        self.fused_append = fused
        self._bind_append()

    def _bind_append(self):
        # decode args that also append (kept apart from the plain ones, which run_step uses)
        self.append_decode_args = {}
        if not getattr(self, "fused_append", False):
            return
        for l in self.layers:
            a = tg.tg_decode_args.from_buffer_copy(self.dplans[l].args)
            a.append_k, a.append_v = self.k_tok[l].data_ptr(), self.v_tok[l].data_ptr()
            a.append_full = self.full.data_ptr()
            self.append_decode_args[l] = a

    def append_layer(self, l, stream=None):
        tg.tg_append(self.append_args[l], stream)

    def run_decode_step(self, stream=None):
        """One decode step: per layer, the new token's K/V appended, then attention over the cache."""
        for l in self.layers:
            if self.fused_append:
                tg.tg_decode(self.append_decode_args[l], stream)
            else:
                tg.tg_append(self.append_args[l], stream)
                tg.tg_decode(self.dplans[l].args, stream)

    def run_layer(self, l, stream=None):
        tg.tg_decode(self.dplans[l].args, stream)

    def run_step(self, stream=None):
        for l in self.layers:
            tg.tg_decode(self.dplans[l].args, stream)

    def capture_step(self, stream):
        """Captures one step (every layer's decode and merge launches) into a HIP graph on
        `stream`; replaying it re-runs the step with the same buffers."""
        graph = torch.cuda.CUDAGraph()
        stream.synchronize()
        with torch.cuda.graph(graph, stream=stream):
            self.run_step(stream)
        return graph

    def stamp_layer(self, l, stream=None):
        """Runs layer l's decode once with per-worker stamps: [n_bins][2] start / end s_memrealtime
        ticks (REALTIME_HZ), as float64 on the host."""
        dp = self.dplans[l]
        ts = torch.zeros(2 * dp.host["num_bins"], dtype=torch.int64, device=self.device)
        args = tg.tg_decode_args.from_buffer_copy(dp.args)
        args.timestamps = ts.data_ptr()
        tg.tg_decode(args, stream)
        torch.cuda.synchronize()
        return ts.view(-1, 2).cpu().numpy().astype(np.float64)

    def bin_pages(self, l):
        """Pages every bin of layer l's plan reads (0 for empty bins)."""
        nb = self.plans[l]["bin_offsets"].shape[0] - 1
        npages = -(-self.item_tokens(l) // self.wl.geom.page_size)
        bo = self.plans[l]["bin_offsets"]
        per_bin = np.add.reduceat(npages, bo[:-1]).astype(np.float64) if len(npages) else np.zeros(nb)
        per_bin[np.diff(bo) == 0] = 0
        return per_bin

    def set_bin_weights(self, weights):
        """Rebuilds the sequential-fill plans with bin weights: one int32 array for every layer, a
        dict of per-layer arrays, or None for equal bins."""
        assert self.mode == tg.TG_PLAN_AOT_FILL, "bin weights apply to the sequential-fill plan"
        self.bin_weights = weights
        self._build_plans()
        self._bind()
        self._bind_append()

    def worker_timeline(self, stream=None):
        """Runs one step with per-worker start/end stamps (s_memrealtime ticks) and returns, per layer,
        a dict over the workers that had work, in microseconds: busy_max and busy_mean (end - start),
        ramp (last start - first start), tail (last end - first end), span (last end - first start)."""
        res = []
        for l in self.layers:
            t = self.stamp_layer(l, stream)[np.diff(self.plans[l]["bin_offsets"]) > 0]
            us = 1e6 / REALTIME_HZ
            busy = (t[:, 1] - t[:, 0]) * us
            res.append(dict(busy_max=float(busy.max()), busy_mean=float(busy.mean()),
                            ramp=float(t[:, 0].max() - t[:, 0].min()) * us,
                            tail=float(t[:, 1].max() - t[:, 1].min()) * us,
                            span=float(t[:, 1].max() - t[:, 0].min()) * us))
        return res

    def worker_busy(self, stream=None):
        """Per layer, (max, mean) of the workers' busy time in microseconds (see worker_timeline)."""
        return [(r["busy_max"], r["busy_mean"]) for r in self.worker_timeline(stream)]

    def layer_slabs(self, l):
        """(page id, slot) of every page slab layer l's plan reads, in item order: the decode's reads
        without its queries, for the streaming-read ceiling."""
        g = self.wl.geom
        P = g.page_size
        items = self.plans[l]["items"]
        ntok = self.item_tokens(l)
        npg = -(-ntok // P)
        first = items["pt_base"] + items["tok_begin"] // P
        starts = np.repeat(first, npg) + (np.arange(int(npg.sum())) - np.repeat(np.cumsum(npg) - npg, npg))
        pages = self.t.pt_pages[starts].astype(np.int32)
        slots = np.repeat(items["slot"], npg).astype(np.int32)
        return pages, slots

    def bin_load_stats(self, l):
        """Planned time per bin, as token load divided by the bin's relative weight (1 without bin
        weights, so plain tokens): (max, mean)."""
        p = self.plans[l]
        lens = self.item_tokens(l)
        bo = p["bin_offsets"]
        loads = np.zeros(len(bo) - 1, dtype=np.float64)
        np.add.at(loads, np.repeat(np.arange(len(bo) - 1), np.diff(bo)), lens)
        w = self.bin_weights.get(l) if isinstance(self.bin_weights, dict) else self.bin_weights
        if w is not None and self.mode == tg.TG_PLAN_AOT_FILL:
            w = np.asarray(w, dtype=np.float64)
            loads = loads / (w / w.mean())
        return float(loads.max()), float(loads.mean())


# s_memrealtime runs at a constant 100 MHz on MI300-class GPUs
REALTIME_HZ = 100e6


class PrefillSession:
    """Pool, chunk inputs and output of one chunked-prefill workload (one layer)."""

    def __init__(self, wl, tables: Tables = None, layer=0, fill="device", pool=None, device="cuda", schedule=True,
                 hist_len=None):
        from workloads import S_K, S_POOL, S_Q, S_V, device_normal_, host_pool, host_prefill_inputs, page_elems
        g = wl.geom
        assert wl.chunk_len >= 1, "prefill workloads need a chunk length"
        self.wl, self.layer, self.device = wl, layer, device
        self.t = tables if tables is not None else Tables(wl, device=device)
        # retained history rows per (b, l, h): the reserved lengths, or fewer when the
        # tables also reserve room for entries of this and later chunks
        self.hist = self.t.kv_len if hist_len is None else np.ascontiguousarray(hist_len, dtype=np.int32)
        self.dtype = TORCH_DTYPE[wl.dtype]
        B, C = wl.batch, wl.chunk_len
        if pool is not None:
            self.pool = pool
        elif fill == "host":
            self.pool = torch.from_numpy(host_pool(wl, self.t.pool_pages)).to(self.dtype).to(device)
        else:
            self.pool = torch.empty(self.t.pool_pages * page_elems(g), dtype=self.dtype, device=device)
            device_normal_(self.pool, wl, S_POOL, wl.kv_scale)
        self.pool = self.pool.view(self.t.pool_pages, 2, g.heads_per_group, g.page_size, g.head_dim)
        if fill == "host":
            q, k, v = host_prefill_inputs(wl)
            self.q, self.k_new, self.v_new = (torch.from_numpy(x).to(self.dtype).to(device) for x in (q, k, v))
        else:
            self.q = torch.empty(B, C, g.num_q_heads, g.head_dim, dtype=self.dtype, device=device)
            self.k_new = torch.empty(B, C, g.num_kv_heads, g.head_dim, dtype=self.dtype, device=device)
            self.v_new = torch.empty_like(self.k_new)
            device_normal_(self.q, wl, S_Q, wl.q_scale)
            device_normal_(self.k_new, wl, S_K, wl.kv_scale)
            device_normal_(self.v_new, wl, S_V, wl.kv_scale)
        self.out = torch.zeros(B, C, g.num_q_heads, g.head_dim, dtype=self.dtype, device=device)
        self.d_offsets = to_device(self.t.pt_offsets, device)
        self.d_kv_len = to_device(self.hist, device)
        self.d_group_of = to_device(self.t.group_of, device)
        self.d_slot_of = to_device(self.t.slot_of, device)
        # ahead-of-time workgroup schedule from the retained lengths (host integer work)
        self.order = tg.tg_prefill_schedule(g, B, C, layer, self.hist) if schedule else None
        self.d_order = to_device(self.order, device) if schedule else None
        self.args = tg.make_prefill_args(g, B, C, layer, TG_DTYPE[wl.dtype], self.q, self.k_new, self.v_new,
                                         self.pool, self.t.d_pt_pages, self.d_offsets, self.d_kv_len,
                                         self.d_group_of, self.d_slot_of, self.out, block_order=self.d_order)

    def run(self, stream=None):
        tg.tg_prefill(self.args, stream)

    def min_hbm_bytes(self) -> int:
        """Bytes one launch must move at least: Q, each KV head's retained history and chunk K/V read once,
        the output written once."""
        g, wl = self.wl.geom, self.wl
        esz = self.q.element_size()
        B, C, d = wl.batch, wl.chunk_len, g.head_dim
        hist = int(self.hist[:, self.layer, :].astype(np.int64).sum())
        return int(esz * d * (2 * B * C * g.num_q_heads + 2 * B * C * g.num_kv_heads + 2 * hist))

    def flops(self) -> int:
        """Algorithmic flops: 4*d per (query row, visible key) for q.k and p.v."""
        g, wl = self.wl.geom, self.wl
        C = wl.chunk_len
        hist = self.hist[:, self.layer, :].astype(np.int64)              # [B][H]
        per_row_keys = hist.sum() * C + wl.batch * g.num_kv_heads * C * (C + 1) // 2
        return int(4 * g.head_dim * g.gqa * per_row_keys)


class CompressSession:
    """One prefill chunk's compression into the ragged cache (one layer), on the GPU.

    `tables` must reserve each request's whole context (the chunk included);
    chunk_start[b] context tokens precede the chunk and chunk_tokens[b] of its
    chunk_len rows are valid.  k_new, v_new [B][C][H][d] and scores [B][H][C]
    are device tensors (drawn from the workload's seeded streams when None).
    The counts and work items come from tg_compress_plan (host, before the
    step); run() enqueues tg_compress."""

    def __init__(self, wl, tables: Tables, pool, chunk_start, chunk_tokens, layer=0, sel_ratio="reserved",
                 rows_per_item=32, k_new=None, v_new=None, scores=None, device="cuda"):
        from workloads import S_K, S_V, device_normal_, host_scores
        g = wl.geom
        B, C, H = wl.batch, wl.chunk_len, g.num_kv_heads
        self.wl, self.t, self.layer, self.device = wl, tables, layer, device
        self.pool = pool
        self.dtype = TORCH_DTYPE[wl.dtype]
        self.chunk_start = np.asarray(chunk_start, dtype=np.int32)
        self.chunk_tokens = np.asarray(chunk_tokens, dtype=np.int32)
        ratio = wl.ratio if isinstance(sel_ratio, str) and sel_ratio == "reserved" else sel_ratio
        t0 = time.perf_counter()
        self.plan = tg.tg_compress_plan(g, B, layer, C, self.chunk_start, self.chunk_tokens, ratio, wl.budget,
                                        tables.kv_len, tables.pt_offsets, tables.group_of, tables.slot_of,
                                        rows_per_item)
        self.plan_us = (time.perf_counter() - t0) * 1e6
        self.d_items = to_device(self.plan["items"] if self.plan["num_items"]
                                 else np.zeros(1, tg.COMPRESS_ITEM_DTYPE), device)
        if k_new is None:
            k_new = torch.empty(B, C, H, g.head_dim, dtype=self.dtype, device=device)
            v_new = torch.empty_like(k_new)
            device_normal_(k_new, wl, S_K, wl.kv_scale)
            device_normal_(v_new, wl, S_V, wl.kv_scale)
        self.k_new, self.v_new = k_new, v_new
        self.scores = scores if scores is not None else torch.from_numpy(host_scores(wl, (B, H, C))).to(device)
        self.d_chunk_tokens = to_device(self.chunk_tokens, device)
        self.d_keep_count = to_device(self.plan["keep_count"], device)
        self.kept = torch.full((B, H, C), -1, dtype=torch.int32, device=device)
        self.args = tg.make_compress_args(g, B, C, TG_DTYPE[wl.dtype], self.k_new, self.v_new, self.scores,
                                          self.pool, tables.d_pt_pages, self.d_items, self.plan["num_items"],
                                          self.d_chunk_tokens, self.d_keep_count, self.kept)

    def run(self, stream=None):
        tg.tg_compress(self.args, stream)

    def traffic_bytes(self) -> int:
        """Algorithmic HBM bytes of one call: the kept K and V rows read from the chunk and
        written to the pages, the valid scores read once, and the kept indices written once
        (and read back by the copy)."""
        g = self.wl.geom
        esz = 4 if self.wl.dtype == "f32" else 2
        kept = int(self.plan["keep_count"].sum())
        scores = int(self.chunk_tokens.astype(np.int64).sum()) * g.num_kv_heads * 4
        return kept * 2 * g.head_dim * esz * 2 + scores + kept * 4 * 2
