"""Ragged chunked-prefill attention (bf16 MFMA kernel, through the C ABI) vs the fp64 oracle."""
import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import check_close, poisoned_host_pool, say, sweep_cases
from workloads import Geometry, config, custom

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from paper_2606_06302_amd.runner import PrefillSession, Tables


def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _oracle(ps, rows):
    """fp64 oracle for the given (b, q_head) rows, from pages copied back."""
    wl, t = ps.wl, ps.t
    g = wl.geom
    L, G, P = g.num_layers, g.num_groups, g.page_size
    need = []
    for b, qh in rows:
        h = qh // g.gqa
        base = int(t.pt_offsets[(b * L + ps.layer) * G + t.group_of[ps.layer, h]])
        need.append(t.pt_pages[base: base + (int(ps.hist[b, ps.layer, h]) + P - 1) // P])
    idx = np.unique(np.concatenate(need + [np.zeros(1, dtype=np.int64)])).astype(np.int64)
    sub = ps.pool[torch.from_numpy(idx).cuda()].float().cpu().numpy().astype(np.float64)
    remap = np.full(t.pool_pages, -1, dtype=np.int64)
    remap[idx] = np.arange(len(idx))
    f = lambda x: x.float().cpu().numpy().astype(np.float64)
    return oracle.prefill_attention(f(ps.q), f(ps.k_new), f(ps.v_new), sub, ps.layer, geom=g, kv_len=ps.hist,
                                    offsets=t.pt_offsets, pages=remap[t.pt_pages], group_of=t.group_of,
                                    slot_of=t.slot_of, rows=rows)


def _compare(ps, rows, what):
    ref = _oracle(ps, rows)
    got = ps.out.float().cpu().numpy().astype(np.float64)
    bi = [r[0] for r in rows]
    qi = [r[1] for r in rows]
    g = np.stack([got[b, :, q] for b, q in zip(bi, qi)])
    r = np.stack([ref[b, :, q] for b, q in zip(bi, qi)])
    return check_close(g.reshape(-1, g.shape[-1]), r.reshape(-1, r.shape[-1]), "bf16", what)


@pytest.mark.parametrize("d", [128, 64])
@pytest.mark.parametrize("gqa,C,Hp,ctx", [(4, 40, 2, 300), (1, 33, 1, 100), (3, 70, 2, (20, 600)), (8, 128, 4, 1000),
                                          (16, 9, 2, 50), (2, 1, 1, 64), (5, 200, 1, (1, 2000))])
def test_prefill_small_vs_oracle(gqa, C, Hp, ctx, d):
    _gpu()
    H = 4 if Hp != 1 else 2
    g = Geometry(1, H, H * gqa, d, 16, Hp)
    wl = custom(500 + gqa * 7 + C + d, g, 3, "bf16", ctx, chunk_len=C)
    say(f"prefill d={d} gqa={gqa} C={C} Hp={Hp} ctx={wl.ctx_len.tolist()}")
    tables = Tables(wl)
    pool = torch.from_numpy(poisoned_host_pool(wl, tables)).to(torch.bfloat16).cuda()
    ps = PrefillSession(wl, tables=tables, fill="host", pool=pool)
    ps.run()
    torch.cuda.synchronize()
    rows = [(b, q) for b in range(wl.batch) for q in range(g.num_q_heads)]
    _compare(ps, rows, f"gqa {gqa} C {C}")


@pytest.mark.parametrize("d", [128, 64])
def test_prefill_short_and_empty_histories(d):
    """Histories shorter than the reservation, down to none at all (a prompt's first chunk): heads with 0,
    1, 15, 16, 17 and 63 retained rows and one with its whole reservation, NaN in every pool row past them."""
    _gpu()
    g = Geometry(1, 8, 32, d, 16, 2)
    wl = custom(640, g, 3, "bf16", (200, 900), chunk_len=77)
    tables = Tables(wl)
    pool = torch.from_numpy(poisoned_host_pool(wl, tables)).to(torch.bfloat16).cuda()
    hist = np.minimum(tables.kv_len, np.array([0, 1, 15, 16, 17, 63, 10**6, 0], dtype=np.int32)[None, None, :])
    hist[1] = 0                                   # a request with no history in any head
    say(f"prefill short histories {hist[:, 0].tolist()}")
    ps = PrefillSession(wl, tables=tables, fill="host", pool=pool, hist_len=hist)
    ps.run()
    torch.cuda.synchronize()
    _compare(ps, [(b, q) for b in range(wl.batch) for q in range(g.num_q_heads)], "short histories")


def test_prefill_history_lengths_are_clamped_to_the_table():
    """A history length past the head's table, or below zero, is clamped to [0, pages * page_size] on the
    device: the output equals the oracle's over the clamped lengths."""
    _gpu()
    g = Geometry(1, 8, 32, 128, 16, 2)
    wl = custom(652, g, 2, "bf16", (100, 700), chunk_len=40)
    tables = Tables(wl)
    L, G, P = g.num_layers, g.num_groups, g.page_size
    cap = np.zeros_like(tables.kv_len)
    for b in range(wl.batch):
        for h in range(g.num_kv_heads):
            t = (b * L) * G + int(tables.group_of[0, h])
            cap[b, 0, h] = (int(tables.pt_offsets[t + 1]) - int(tables.pt_offsets[t])) * P
    raw = tables.kv_len.copy()
    raw[0, 0, :4] = cap[0, 0, :4] + np.array([1, 16, 1000, 2 ** 30])
    raw[1, 0, 0] = -5
    raw[1, 0, 1] = np.iinfo(np.int32).min
    say(f"prefill raw lengths {raw[:, 0].tolist()} capacity {cap[:, 0].tolist()}")
    # every reserved row holds data here: clamping to the capacity makes rows past kv_len part of the history
    ps = PrefillSession(wl, tables=tables, fill="host", hist_len=raw, schedule=False)
    ps.run()
    torch.cuda.synchronize()
    ps.hist = np.clip(raw, 0, cap).astype(np.int32)   # what the oracle is given
    _compare(ps, [(b, q) for b in range(wl.batch) for q in range(g.num_q_heads)], "clamped lengths")


def test_prefill_long_chunk_sampled():
    """A 4096-token chunk at gqa 8 (32768 query rows per unit, 128 row tiles, 64 chunk tiles): sampled
    (request, query head) rows over every chunk position against the oracle."""
    _gpu()
    g = Geometry(1, 4, 32, 128, 16, 2)
    wl = custom(661, g, 2, "bf16", (500, 3000), chunk_len=4096)
    say(f"prefill long chunk C={wl.chunk_len} gqa={g.gqa} ctx={wl.ctx_len.tolist()}")
    tables = Tables(wl)
    pool = torch.from_numpy(poisoned_host_pool(wl, tables)).to(torch.bfloat16).cuda()
    ps = PrefillSession(wl, tables=tables, fill="host", pool=pool)
    ps.run()
    torch.cuda.synchronize()
    rows = [(0, 0), (0, 13), (1, 31)]
    rows.append((int(np.argmax(tables.kv_len[:, 0].max(axis=1))), int(np.argmax(tables.kv_len[:, 0].max(axis=0))) * g.gqa))
    _compare(ps, sorted(set(rows)), "long chunk")


@pytest.mark.parametrize("plan", ["fill", "aot"])
def test_prefill_chunk_of_one_matches_decode_path(plan):
    """C = 1: one chunk row of chunked prefill (Section 2.2.1) sees exactly what the split-KV decode path
    (Section 2.2.3) sees once the chunk's key and value are the cache's next entry.  The prefill kernel runs
    over the history; then tg_append writes the chunk's K and V as entry kv_len of every head (into a row that
    holds NaN until then) and the decode kernel, on an open-ended plan, attends over kv_len + 1 entries with the
    same queries.  Both outputs match the oracle and each other within the bf16 tolerance."""
    _gpu()
    from paper_2606_06302_amd import tangram as tg
    from paper_2606_06302_amd.runner import DecodeSession
    g = Geometry(1, 8, 32, 128, 16, 2)
    wl = custom(612, g, 4, "bf16", (100, 900), chunk_len=1)
    tables = Tables(wl, headroom=np.ones(wl.batch, dtype=np.int32))
    pool = torch.from_numpy(poisoned_host_pool(wl, tables)).to(torch.bfloat16).cuda()
    say(f"C=1 vs decode ({plan}): ctx={wl.ctx_len.tolist()}")
    ps = PrefillSession(wl, tables=tables, fill="host", pool=pool)
    ps.run()
    torch.cuda.synchronize()
    rows = [(b, q) for b in range(wl.batch) for q in range(g.num_q_heads)]
    _compare(ps, rows, "C=1 prefill")

    mode = tg.TG_PLAN_AOT_FILL if plan == "fill" else tg.TG_PLAN_AOT
    q = ps.q[:, 0].unsqueeze(0).contiguous()                     # [L=1][B][Hq][d]
    ds = DecodeSession(wl, tables=tables, mode=mode, n_bins=29, split_target=40, fill="host", pool=pool, q=q,
                       open_end=True)
    ds.enable_append(k_tok=ps.k_new[:, 0].unsqueeze(0).contiguous(), v_tok=ps.v_new[:, 0].unsqueeze(0).contiguous())
    ds.run_decode_step()                                         # append, then attend
    torch.cuda.synchronize()
    assert int(ds.full.item()) == 0
    assert np.array_equal(ds.live_len.cpu().numpy(), tables.kv_len + 1)
    # the decode over kv_len + 1 entries against the oracle (the pool as the append left it)
    f = lambda x: x.float().cpu().numpy().astype(np.float64)
    t = tables
    O, _ = oracle.decode_attention(f(q[0]), f(ds.pool), 0, geom=g, batch=wl.batch, kv_len=t.kv_len + 1,
                                   offsets=t.pt_offsets, pages=t.pt_pages, group_of=t.group_of, slot_of=t.slot_of)
    dec = f(ds.out[0])
    check_close(dec.reshape(-1, g.head_dim), O.reshape(-1, g.head_dim), "bf16", "C=1 decode vs oracle")
    pre = f(ps.out[:, 0])
    check_close(dec.reshape(-1, g.head_dim), pre.reshape(-1, g.head_dim), "bf16", "C=1 decode vs prefill")


def test_prefill_config5_full_size_sampled():
    _gpu()
    wl = config(5)
    say(f"config 5 full size: B={wl.batch} C={wl.chunk_len}")
    ps = PrefillSession(wl)
    ps.run()
    torch.cuda.synchronize()
    rng = np.random.default_rng(55)
    rows = [(int(rng.integers(0, wl.batch)), int(rng.integers(0, wl.geom.num_q_heads))) for _ in range(6)]
    b = int(np.argmax(ps.t.kv_len[:, 0, :].max(axis=1)))
    rows.append((b, int(np.argmax(ps.t.kv_len[b, 0])) * wl.geom.gqa))      # the longest history
    _compare(ps, sorted(set(rows)), "config 5")


def test_prefill_block_order_does_not_change_results():
    """The ahead-of-time schedule only reorders workgroups: outputs are bitwise
    equal with the default mapping and with schedules for 8 and 3 XCDs."""
    _gpu()
    from paper_2606_06302_amd import tangram as tg
    from paper_2606_06302_amd.device import to_device
    g = Geometry(1, 8, 32, 128, 16, 2)
    wl = custom(733, g, 5, "bf16", (50, 3000), chunk_len=300)
    tables = Tables(wl)
    pool = torch.from_numpy(poisoned_host_pool(wl, tables)).to(torch.bfloat16).cuda()
    ps = PrefillSession(wl, tables=tables, fill="host", pool=pool, schedule=False)
    ps.run()
    torch.cuda.synchronize()
    base = ps.out.clone()
    for n_xcd in (8, 3):
        order = to_device(tg.tg_prefill_schedule(g, wl.batch, wl.chunk_len, 0, tables.kv_len, n_xcd), "cuda")
        say(f"block order n_xcd={n_xcd}: {order.numel()} blocks")
        ps.out.zero_()
        args = tg.make_prefill_args(g, wl.batch, wl.chunk_len, 0, tg.TG_BF16, ps.q, ps.k_new, ps.v_new, ps.pool,
                                    tables.d_pt_pages, ps.d_offsets, ps.d_kv_len, ps.d_group_of, ps.d_slot_of,
                                    ps.out, block_order=order)
        tg.tg_prefill(args)
        torch.cuda.synchronize()
        assert torch.equal(ps.out, base)
    _compare(ps, [(b, q) for b in range(wl.batch) for q in range(0, 32, 3)], "scheduled")


def test_prefill_random_shapes_sweep():
    """Seeded sweep: 10 random (head_dim, gqa, KV heads, heads per group, batch, chunk length, context range) cases,
    every (request, query head) row against the oracle, NaN past the retained history."""
    _gpu()
    rng = np.random.default_rng(777)
    for case in range(sweep_cases(10)):
        gqa = int(rng.integers(1, 17))
        H = [1, 2, 4, 8][int(rng.integers(4))]
        Hp = [x for x in (1, 2, 4) if H % x == 0][int(rng.integers(len([x for x in (1, 2, 4) if H % x == 0])))]
        B = int(rng.integers(1, 4))
        C = int(rng.integers(1, 301))
        lo = int(rng.integers(1, 300))
        hi = lo + int(rng.integers(0, 1500))
        d = [64, 128][int(rng.integers(2))]
        g = Geometry(1, H, H * gqa, d, 16, Hp)
        wl = custom(7000 + case, g, B, "bf16", (lo, hi) if hi > lo else lo, chunk_len=C)
        say(f"prefill sweep case {case}: d{d} gqa{gqa} H{H} Hp{Hp} B{B} C{C} ctx={wl.ctx_len.tolist()}")
        tables = Tables(wl)
        pool = torch.from_numpy(poisoned_host_pool(wl, tables)).to(torch.bfloat16).cuda()
        ps = PrefillSession(wl, tables=tables, fill="host", pool=pool)
        ps.run()
        torch.cuda.synchronize()
        _compare(ps, [(b, q) for b in range(B) for q in range(g.num_q_heads)], f"prefill sweep case {case}")
