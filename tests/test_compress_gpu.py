"""Compression of a prefill chunk into the ragged cache (tg_compress, through the C ABI) vs the oracle.

The kernel only selects and copies, so the bar is bit-exact: the whole pool
after the call (kept rows written, every other row untouched) and the kept
index lists must equal the oracle's.
"""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import compare_layer, say, sweep_cases
from workloads import Geometry, config, custom, host_pool, host_scores

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from paper_2606_06302_amd.runner import TORCH_DTYPE, CompressSession, DecodeSession, Tables


def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _f64(t):
    return t.float().cpu().numpy().astype(np.float64)


def _run_and_check(wl, tables, pool, starts, toks, sel, R, layer, rng, special=True):
    """One chunk: tg_compress on the device pool, the oracle on a host copy; both compared in full."""
    g = wl.geom
    B, C, H, d = wl.batch, wl.chunk_len, g.num_kv_heads, g.head_dim
    dt = TORCH_DTYPE[wl.dtype]
    k = torch.from_numpy(rng.standard_normal((B, C, H, d), dtype=np.float32)).to(dt).cuda()
    v = torch.from_numpy(rng.standard_normal((B, C, H, d), dtype=np.float32)).to(dt).cuda()
    sc = host_scores(dataclasses.replace(wl, seed=int(rng.integers(1 << 30))), (B, H, C), special=special)
    before = _f64(pool)
    cs = CompressSession(wl, tables, pool, starts, toks, layer=layer, sel_ratio=sel, rows_per_item=R, k_new=k,
                         v_new=v, scores=torch.from_numpy(sc).cuda())
    cs.run()
    torch.cuda.synchronize()
    sel_r = wl.ratio if isinstance(sel, str) else sel
    ref, kept, cur, cnt = oracle.compress_chunk(_f64(k), _f64(v), sc, before, layer, geom=g, ratio=sel_r,
                                                capacity=tables.kv_len, chunk_start=starts, chunk_tokens=toks,
                                                offsets=tables.pt_offsets, pages=tables.pt_pages,
                                                group_of=tables.group_of, slot_of=tables.slot_of)
    assert np.array_equal(cs.plan["write_begin"], cur) and np.array_equal(cs.plan["keep_count"], cnt)
    got = _f64(pool)
    bad = np.argwhere(got != ref)
    assert len(bad) == 0, f"{len(bad)} pool elements differ, first {bad[:3].tolist()}"
    kept_dev = cs.kept.cpu().numpy()
    for b in range(B):
        for h in range(H):
            n = int(cnt[b, h])
            assert kept_dev[b, h, :n].tolist() == kept[b][h], (b, h)
            assert (kept_dev[b, h, n:] == -1).all(), (b, h)
    return cs, int(cnt.sum())


def _pool_for(wl, tables):
    return torch.from_numpy(host_pool(wl, tables.pool_pages)).to(TORCH_DTYPE[wl.dtype]).cuda().view(
        tables.pool_pages, 2, wl.geom.heads_per_group, wl.geom.page_size, wl.geom.head_dim)


CASES = [
    # (geometry, batch, dtype, chunk_len, rows_per_item, selection ratio, layer, fixed budgets)
    (Geometry(1, 4, 8, 64, 16, 2), 3, "f32", 37, 5, "reserved", 0, None),
    (Geometry(1, 8, 32, 128, 16, 2), 4, "bf16", 512, 64, "reserved", 0, None),
    (Geometry(1, 2, 2, 64, 16, 1), 2, "bf16", 1, 1, "reserved", 0, [[1.0, 0.5]]),
    (Geometry(1, 8, 8, 128, 16, 4), 2, "f32", 300, 256, "overflow", 0, None),
    (Geometry(2, 4, 16, 128, 16, 2), 3, "bf16", 2000, 64, "reserved", 1, None),
    (Geometry(1, 4, 4, 64, 5, 2), 2, "bf16", 100, 7, "overflow", 0, None),
    (Geometry(1, 4, 8, 128, 16, 2), 2, "bf16", 200, 32, "reserved", 0, None),
    (Geometry(1, 2, 4, 128, 16, 1), 2, "f32", 1024, 256, "overflow", 0, None),
]


@pytest.mark.parametrize("geom,B,dtype,C,R,sel,layer,budget", CASES)
def test_compress_small_vs_oracle(geom, B, dtype, C, R, sel, layer, budget):
    _gpu()
    seed = 800 + C + R + B
    rng = np.random.default_rng(seed)
    ctx = rng.integers(C, 4 * C + 20, size=B).astype(np.int32)
    wl = custom(seed, geom, B, dtype, ctx, chunk_len=C, budget=budget, jitter=0.0 if budget else 0.03)
    # ragged chunks anywhere in the context, including an empty one and a full one
    toks = np.array([C, 0] + [int(rng.integers(1, C + 1)) for _ in range(B - 2)], dtype=np.int32)[:B]
    starts = np.array([int(rng.integers(0, c - n + 1)) for c, n in zip(ctx, toks)], dtype=np.int32)
    sel_r = np.minimum(1.0, wl.ratio * 1.7) if sel == "overflow" else "reserved"
    say(f"compress {geom} B={B} {dtype} C={C} R={R} sel={sel} starts={starts.tolist()} toks={toks.tolist()}")
    tables = Tables(wl)
    pool = _pool_for(wl, tables)
    _, kept = _run_and_check(wl, tables, pool, starts, toks, sel_r, R, layer, rng)
    assert kept > 0


@pytest.mark.parametrize("C", [64, 65, 128, 129, 256, 257, 1023, 1024, 1025, 4096, 4097])
def test_compress_chunk_lengths_at_kernel_boundaries(C):
    """Chunk lengths on both sides of the one-launch kernel's keys-per-lane steps (64, 128, 256 tokens), of
    the one-launch limit (1024) and of the select launch's switch from 512 to 1024 threads (4096): the whole
    pool and the kept lists bit-exact against the oracle, with ties, signed zeros, infinities and NaN among
    the scores."""
    _gpu()
    g = Geometry(1, 4, 16, 128, 16, 2)
    B = 3
    rng = np.random.default_rng(4000 + C)
    ctx = rng.integers(C, 3 * C + 20, size=B).astype(np.int32)
    wl = custom(4000 + C, g, B, "bf16", ctx, chunk_len=C)
    toks = np.array([C, int(rng.integers(1, C + 1)), max(1, C - 1)], dtype=np.int32)
    starts = np.array([int(rng.integers(0, c - n + 1)) for c, n in zip(ctx, toks)], dtype=np.int32)
    say(f"compress boundary C={C} toks={toks.tolist()}")
    tables = Tables(wl)
    pool = _pool_for(wl, tables)
    _, kept = _run_and_check(wl, tables, pool, starts, toks, np.minimum(1.0, wl.ratio * 1.3), 32, 0, rng)
    assert kept > 0


def test_compress_three_chunks_then_decode():
    """A context compressed chunk by chunk fills its reservation exactly; decode attention over the
    resulting cache matches the oracle (prefill compression feeding the decode kernel)."""
    _gpu()
    g = Geometry(1, 8, 32, 128, 16, 2)
    B, C = 3, 700
    ctx = np.full(B, 3 * C, dtype=np.int32)
    wl = custom(901, g, B, "bf16", ctx, chunk_len=C)
    tables = Tables(wl)
    pool = _pool_for(wl, tables)
    rng = np.random.default_rng(901)
    for c in range(3):
        say(f"chunk {c}")
        _run_and_check(wl, tables, pool, np.full(B, c * C), np.full(B, C), "reserved", 64, 0, rng)
    s = DecodeSession(wl, tables=tables, pool=pool.view(-1), fill="host", n_bins=64, split_target=128)
    s.run_step()
    torch.cuda.synchronize()
    compare_layer(s, 0, what="decode after chunked compression")


def test_compress_longest_chunk():
    """chunk_len at TG_COMPRESS_MAX_CHUNK: the 64 KiB LDS key buffer."""
    _gpu()
    from paper_2606_06302_amd import tangram as tg
    g = Geometry(1, 2, 2, 128, 16, 2)
    C = tg.TG_COMPRESS_MAX_CHUNK
    wl = custom(933, g, 1, "bf16", [C], budget=np.array([[0.5, 0.03]]), jitter=0.0, chunk_len=C)
    tables = Tables(wl)
    pool = _pool_for(wl, tables)
    _run_and_check(wl, tables, pool, [0], [C], "reserved", 256, 0, np.random.default_rng(933))


def test_compress_config5_chunk_full_size():
    """Config 5's chunk (512 tokens after a 16384-token history, 16 requests, 8 KV heads, bf16), in the
    launch configuration the benchmark times: kept lists equal the oracle's, every kept row lands at
    its entry, and no other row of the pool changes."""
    _gpu()
    wl5 = config(5)
    C = wl5.chunk_len
    wl = dataclasses.replace(wl5, ctx_len=wl5.ctx_len + C)
    g = wl.geom
    tables = Tables(wl)
    from workloads import S_POOL, device_normal_, page_elems
    pool = torch.empty(tables.pool_pages * page_elems(g), dtype=torch.bfloat16, device="cuda")
    device_normal_(pool, wl, S_POOL, wl.kv_scale)
    pool = pool.view(tables.pool_pages, 2, g.heads_per_group, g.page_size, g.head_dim)
    before = pool.clone()
    cs = CompressSession(wl, tables, pool, wl5.ctx_len, np.full(wl.batch, C))
    say(f"config 5 chunk: {cs.plan['num_items']} items, {int(cs.plan['keep_count'].sum())} kept rows")
    cs.run()
    torch.cuda.synchronize()
    sc = cs.scores.cpu().numpy()
    kept_dev = cs.kept.cpu().numpy()
    L, G, P = g.num_layers, g.num_groups, g.page_size
    written = torch.zeros(pool.shape[:4], dtype=torch.bool, device="cuda")
    for b in range(wl.batch):
        for h in range(g.num_kv_heads):
            cur, cnt = int(cs.plan["write_begin"][b, h]), int(cs.plan["keep_count"][b, h])
            want = oracle.top_entries(sc[b, h], cnt)
            assert kept_dev[b, h, :cnt].tolist() == want, (b, h)
            base = int(tables.pt_offsets[(b * L) * G + tables.group_of[0, h]])
            pos = np.arange(cur, cur + cnt)
            pages = torch.from_numpy(tables.pt_pages[base + pos // P].astype(np.int64)).cuda()
            rows = torch.from_numpy(pos % P).cuda()
            s = int(tables.slot_of[0, h])
            idx = torch.tensor(want, dtype=torch.int64, device="cuda")
            assert torch.equal(pool[pages, 0, s, rows], cs.k_new[b, idx, h])
            assert torch.equal(pool[pages, 1, s, rows], cs.v_new[b, idx, h])
            written[pages, :, s, rows] = True
    changed = (pool != before).any(dim=-1)
    assert not bool((changed & ~written).any())


def test_compress_random_sweep():
    """Seeded sweep: 8 random (dtype, head_dim, KV heads, heads per group, batch, chunk length, rows per item,
    selection ratio) cases, each chunk placed anywhere in its context; the whole pool and the kept lists
    bit-exact against the oracle."""
    _gpu()
    rng = np.random.default_rng(9090)
    for case in range(sweep_cases(8)):
        dtype = ["f32", "bf16"][int(rng.integers(2))]
        d = [64, 128][int(rng.integers(2))]
        H = [1, 2, 4, 8][int(rng.integers(4))]
        Hp = [x for x in (1, 2, 4, 8) if H % x == 0][int(rng.integers(len([x for x in (1, 2, 4, 8) if H % x == 0])))]
        B = int(rng.integers(1, 5))
        C = int(rng.integers(1, 2001))
        R = int(rng.integers(1, 257))
        g = Geometry(1, H, H * 2, d, 16, Hp)
        ctx = rng.integers(C, 3 * C + 50, size=B).astype(np.int32)
        wl = custom(9100 + case, g, B, dtype, ctx, chunk_len=C)
        toks = rng.integers(0, C + 1, size=B).astype(np.int32)
        starts = np.array([int(rng.integers(0, c - n + 1)) for c, n in zip(ctx, toks)], dtype=np.int32)
        sel = np.minimum(1.0, wl.ratio * 1.5) if case % 2 else "reserved"
        say(f"compress sweep case {case}: {dtype} d{d} H{H} Hp{Hp} B{B} C{C} R{R} "
            f"{'overflow' if case % 2 else 'reserved'} starts={starts.tolist()} toks={toks.tolist()}")
        tables = Tables(wl)
        pool = _pool_for(wl, tables)
        _run_and_check(wl, tables, pool, starts, toks, sel, R, 0, rng)
