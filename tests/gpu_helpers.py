"""Test-side helpers for the GPU parity tests: poisoning, sampled oracle runs, tolerances."""
from __future__ import annotations

import math
import os
import sys

import numpy as np
import torch

import oracle

# Tolerances: bf16 max abs 2e-2 plus a relative L2 bound (outputs of diffuse
# attention are small, so an absolute bound alone would accept a zero output);
# fp32 max abs 1e-4.
TOL = {"f32": dict(atol=1e-4, rel=1e-4), "bf16": dict(atol=2e-2, rel=1e-2)}
LSE_TOL = {"f32": 1e-4, "bf16": 2e-3}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def retained_mask(tables, wl):
    """Boolean [pool_pages][2][H_p][P] marking rows that hold a retained entry."""
    g = wl.geom
    P, G, L, H = g.page_size, g.num_groups, g.num_layers, g.num_kv_heads
    mask = np.zeros((tables.pool_pages, 2, g.heads_per_group, P), dtype=bool)
    for b in range(wl.batch):
        for l in range(L):
            for h in range(H):
                n = int(tables.kv_len[b, l, h])
                base = int(tables.pt_offsets[(b * L + l) * G + tables.group_of[l, h]])
                s = int(tables.slot_of[l, h])
                pages = tables.pt_pages[base: base + (n + P - 1) // P]
                full = n // P
                mask[pages[:full], :, s, :] = True
                if n % P:
                    mask[pages[full], :, s, : n % P] = True
    return mask


def poisoned_host_pool(wl, tables):
    """Seeded N(0, s^2) pool whose rows outside any retained entry are NaN."""
    from workloads import host_pool
    g = wl.geom
    pool = host_pool(wl, tables.pool_pages).reshape(tables.pool_pages, 2, g.heads_per_group, g.page_size,
                                                     g.head_dim)
    pool[~retained_mask(tables, wl)] = np.nan
    return pool


def compact_pool(session, layer, pairs):
    """Copies only the pages the given (b, kv_head) pairs read; returns (pool64, remapped pages)."""
    t, g, wl = session.t, session.wl.geom, session.wl
    L, G, P = g.num_layers, g.num_groups, g.page_size
    need = []
    for b, h in pairs:
        base = int(t.pt_offsets[(b * L + layer) * G + t.group_of[layer, h]])
        n = int(t.kv_len[b, layer, h])
        need.append(t.pt_pages[base: base + (n + P - 1) // P])
    idx = np.unique(np.concatenate(need)).astype(np.int64)
    sub = session.pool[torch.from_numpy(idx).to(session.pool.device)].float().cpu().numpy().astype(np.float64)
    remap = np.full(session.t.pool_pages, -1, dtype=np.int64)
    remap[idx] = np.arange(len(idx))
    return sub, remap[t.pt_pages]


def oracle_decode(session, layer, pairs=None, sm_scale=0.0):
    """fp64 oracle output for one layer (optionally only for some (b, kv_head) pairs)."""
    wl, t = session.wl, session.t
    if pairs is None:
        pairs = [(b, h) for b in range(wl.batch) for h in range(wl.geom.num_kv_heads)]
    pool, pages = compact_pool(session, layer, pairs)
    q = session.q[layer].float().cpu().numpy().astype(np.float64)
    return oracle.decode_attention(q, pool, layer, geom=wl.geom, batch=wl.batch, kv_len=t.kv_len,
                                   offsets=t.pt_offsets, pages=pages, group_of=t.group_of, slot_of=t.slot_of,
                                   sm_scale=sm_scale, heads=pairs)


def rows_of(pairs, gqa):
    return [(b, h * gqa + j) for b, h in pairs for j in range(gqa)]


def check_close(got, ref, dtype, what=""):
    """got, ref: [n][d] arrays (float64).  Returns (max_abs, rel_l2); raises on failure."""
    diff = got - ref
    max_abs = float(np.abs(diff).max()) if diff.size else 0.0
    rel = float(np.linalg.norm(diff) / max(np.linalg.norm(ref), 1e-30))
    tol = TOL[dtype]
    ok = np.all(np.isfinite(got)) and max_abs <= tol["atol"] and rel <= tol["rel"]
    assert ok, f"{what}: max_abs={max_abs:.3g} rel_l2={rel:.3g} (tol {tol}) finite={np.all(np.isfinite(got))}"
    return max_abs, rel


def compare_layer(session, layer, pairs=None, check_lse=True, what=""):
    wl = session.wl
    gqa = wl.geom.gqa
    if pairs is None:
        pairs = [(b, h) for b in range(wl.batch) for h in range(wl.geom.num_kv_heads)]
    O, lse = oracle_decode(session, layer, pairs)
    rows = rows_of(pairs, gqa)
    bi = np.array([r[0] for r in rows])
    qi = np.array([r[1] for r in rows])
    got = session.out[layer].float().cpu().numpy().astype(np.float64)[bi, qi]
    res = check_close(got, O[bi, qi], wl.dtype, what)
    if check_lse and session.lse is not None:
        gl = session.lse[layer].cpu().numpy().astype(np.float64)[bi, qi]
        err = float(np.abs(gl - lse[bi, qi]).max())
        assert err <= LSE_TOL[wl.dtype], f"{what}: lse max err {err}"
    return res


def sample_pairs(wl, n, seed):
    rng = np.random.default_rng(seed)
    allp = [(b, h) for b in range(wl.batch) for h in range(wl.geom.num_kv_heads)]
    pick = rng.choice(len(allp), size=min(n, len(allp)), replace=False)
    return [allp[i] for i in sorted(pick)]


def math_isclose(a, b):
    return math.isclose(a, b, rel_tol=1e-6)


def sweep_cases(default):
    """Case count of a seeded random sweep: `default`, or TG_SWEEP_CASES for a longer campaign (the first
    `default` cases are the same either way)."""
    return int(os.environ.get("TG_SWEEP_CASES", default))
