"""Decode steps through the C ABI: tg_append writes each step's token after every head's entries, and one
open-ended plan built before the first step serves every later step (tg_decode with live lengths).  The same
steps with the append inside the decode launch (tg_decode's append_k / append_v) give the same bits."""
import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import check_close, say, sweep_cases
from workloads import Geometry, custom, host_pool

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from paper_2606_06302_amd import tangram as tg
    from paper_2606_06302_amd.runner import TORCH_DTYPE, DecodeSession, Tables


def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _f64(t):
    return t.float().cpu().numpy().astype(np.float64)


def _session(geom, B, dtype, ctx, T, mode, seed, n_bins=64, fused=False):
    wl = custom(seed, geom, B, dtype, ctx)
    tables = Tables(wl, headroom=np.full(B, T, dtype=np.int32))
    pool = torch.from_numpy(host_pool(wl, tables.pool_pages)).to(TORCH_DTYPE[dtype]).cuda()
    s = DecodeSession(wl, tables=tables, mode=mode, n_bins=n_bins, split_target=2 * n_bins, fill="host", pool=pool,
                      open_end=True)
    s.enable_append(fused=fused)
    return wl, tables, s


def _step_inputs(rng, s, dtype):
    g = s.wl.geom
    shape_tok = (g.num_layers, s.wl.batch, g.num_kv_heads, g.head_dim)
    k = torch.from_numpy(rng.standard_normal(shape_tok, dtype=np.float32)).to(TORCH_DTYPE[dtype])
    v = torch.from_numpy(rng.standard_normal(shape_tok, dtype=np.float32)).to(TORCH_DTYPE[dtype])
    q = torch.from_numpy(rng.standard_normal(tuple(s.q.shape), dtype=np.float32)).to(TORCH_DTYPE[dtype])
    s.k_tok.copy_(k.cuda())
    s.v_tok.copy_(v.cuda())
    s.q.copy_(q.cuda())
    return _f64(k), _f64(v)


@pytest.mark.parametrize("fused", [False, True], ids=["append-launch", "append-in-decode"])
@pytest.mark.parametrize("geom,dtype,mode", [
    (Geometry(2, 8, 32, 128, 16, 2), "bf16", "fill"),
    (Geometry(2, 8, 40, 128, 16, 2), "bf16", "aot"),
    (Geometry(1, 4, 8, 64, 16, 2), "f32", "fill"),
])
def test_steps_with_one_plan_match_oracle(geom, dtype, mode, fused):
    _gpu()
    T, B = 37, 4
    m = tg.TG_PLAN_AOT_FILL if mode == "fill" else tg.TG_PLAN_AOT
    wl, t, s = _session(geom, B, dtype, (20, 900), T, m, 4242 + geom.num_q_heads, fused=fused)
    say(f"decode steps {geom} {dtype} {mode} fused={fused}: ctx {wl.ctx_len.tolist()}, {T} steps")
    rng = np.random.default_rng(99)
    ref_pool = _f64(s.pool)
    live = t.kv_len.copy()
    for step in range(1, T + 1):
        ks, vs = _step_inputs(rng, s, dtype)
        s.run_decode_step()
        for l in range(geom.num_layers):
            ref_pool, live, full = oracle.append_token(ks[l], vs[l], ref_pool, l, geom=geom, live_len=live,
                                                       offsets=t.pt_offsets, pages=t.pt_pages, group_of=t.group_of,
                                                       slot_of=t.slot_of)
            assert full == []
        if step in (1, 16, T):
            torch.cuda.synchronize()
            assert np.array_equal(s.live_len.cpu().numpy(), live)
            assert np.array_equal(_f64(s.pool), ref_pool), f"pool differs after step {step}"
            q = _f64(s.q)
            for l in range(geom.num_layers):
                O, lse = oracle.decode_attention(q[l], ref_pool, l, geom=geom, batch=B, kv_len=live,
                                                 offsets=t.pt_offsets, pages=t.pt_pages, group_of=t.group_of,
                                                 slot_of=t.slot_of)
                got = _f64(s.out[l]).reshape(-1, geom.head_dim)
                check_close(got, O.reshape(-1, geom.head_dim), dtype, f"step {step} layer {l}")
            say(f"  step {step}: ok")
    assert int(s.full.item()) == 0


def test_append_without_room_sets_flag_and_writes_nothing():
    _gpu()
    g = Geometry(1, 4, 8, 64, 16, 2)
    B = 2
    wl = custom(77, g, B, "bf16", [512, 512], budget=np.array([[1.0, 0.5, 0.25, 0.125]]), jitter=0.0)
    t = Tables(wl)           # no headroom: heads 0 (512 of 512) and 2 (128 of 128) are full
    pool = torch.from_numpy(host_pool(wl, t.pool_pages)).to(torch.bfloat16).cuda()
    s = DecodeSession(wl, tables=t, mode=tg.TG_PLAN_AOT_FILL, n_bins=16, fill="host", pool=pool, open_end=True)
    s.enable_append()
    rng = np.random.default_rng(5)
    ks, vs = _step_inputs(rng, s, "bf16")
    before = _f64(s.pool)
    s.append_layer(0)
    torch.cuda.synchronize()
    ref, live, full = oracle.append_token(ks[0], vs[0], before, 0, geom=g, live_len=t.kv_len, offsets=t.pt_offsets,
                                          pages=t.pt_pages, group_of=t.group_of, slot_of=t.slot_of)
    assert sorted(full) == [(0, 0), (0, 2), (1, 0), (1, 2)]
    assert int(s.full.item()) == 1
    assert np.array_equal(s.live_len.cpu().numpy(), live)
    assert np.array_equal(_f64(s.pool), ref)


def test_reused_plan_equals_fresh_plan():
    """After T steps, the open plan built before the first step and a plan built on the grown lengths give
    the same attention (both within tolerance of the oracle, and of each other)."""
    _gpu()
    g = Geometry(1, 8, 64, 128, 16, 2)
    B, T = 8, 50
    wl, t, s = _session(g, B, "bf16", (500, 5000), T, tg.TG_PLAN_AOT_FILL, 515)
    rng = np.random.default_rng(3)
    for _ in range(T):
        _step_inputs(rng, s, "bf16")
        s.run_decode_step()
    torch.cuda.synchronize()
    reused = _f64(s.out[0])
    live = s.live_len.cpu().numpy()
    fresh = tg.tg_build_plan(g, B, 0, live, t.pt_offsets, t.group_of, t.slot_of, tg.TG_PLAN_AOT_FILL, 64)
    from paper_2606_06302_amd.device import bind_decode, upload_plan
    dp = upload_plan(g, B, fresh, "cuda")
    out2 = torch.zeros_like(s.out[0])
    bind_decode(dp, g, B, tg.TG_BF16, s.q[0], s.pool, t.d_pt_pages, out2)
    tg.tg_decode(dp.args)
    torch.cuda.synchronize()
    O, _ = oracle.decode_attention(_f64(s.q[0]), _f64(s.pool), 0, geom=g, batch=B, kv_len=live, offsets=t.pt_offsets,
                                   pages=t.pt_pages, group_of=t.group_of, slot_of=t.slot_of)
    check_close(reused.reshape(-1, 128), O.reshape(-1, 128), "bf16", "reused plan")
    check_close(_f64(out2).reshape(-1, 128), O.reshape(-1, 128), "bf16", "fresh plan")


def _twin_sessions(geom, B, dtype, ctx, mode, seed, headroom, n_bins, merge):
    """Two sessions on the same tables and equal pools: one appends with tg_append, one inside tg_decode."""
    wl = custom(seed, geom, B, dtype, ctx)
    t = Tables(wl, headroom=None if headroom is None else np.full(B, headroom, dtype=np.int32))
    host = torch.from_numpy(host_pool(wl, t.pool_pages)).to(TORCH_DTYPE[dtype])
    pair = []
    for fused in (False, True):
        s = DecodeSession(wl, tables=t, mode=mode, n_bins=n_bins, split_target=2 * n_bins, fill="host",
                          pool=host.clone().cuda(), open_end=True, fused_merge=merge)
        s.enable_append(fused=fused)
        pair.append(s)
    return wl, t, pair


def _same_bits(a, b):
    return torch.equal(a.view(torch.int16) if a.dtype == torch.bfloat16 else a.view(torch.int32),
                       b.view(torch.int16) if b.dtype == torch.bfloat16 else b.view(torch.int32))


@pytest.mark.parametrize("geom,dtype,mode,merge", [
    (Geometry(2, 8, 32, 128, 16, 2), "bf16", "fill", False),   # matrix-core kernel, 4 query heads per KV head
    (Geometry(2, 8, 32, 128, 16, 2), "bf16", "fill", True),    # ... merging split units in the same launch
    (Geometry(1, 4, 64, 128, 16, 2), "bf16", "aot", False),    # 16 query heads per KV head (3-page ring)
    (Geometry(1, 8, 40, 128, 16, 4), "bf16", "aot", True),     # 5 query heads per KV head
    (Geometry(1, 4, 8, 64, 16, 2), "f32", "fill", False),      # generic kernel, fp32, d 64
    (Geometry(1, 4, 16, 64, 16, 1), "bf16", "aot", False),     # generic kernel, bf16, d 64
    (Geometry(1, 2, 4, 128, 16, 2), "f32", "fill", False),     # generic kernel, fp32, d 128
    (Geometry(1, 4, 4, 128, 16, 2), "bf16", "fill", False),    # matrix-core kernel, one query head per KV head
])
def test_append_in_decode_is_bitwise_append_then_decode(geom, dtype, mode, merge):
    """Every step: out, lse, the whole pool and the live lengths equal bit for bit between tg_append +
    tg_decode and tg_decode with the append (contexts from 1 token, steps across page boundaries)."""
    _gpu()
    B, T = 6, 23
    m = tg.TG_PLAN_AOT_FILL if mode == "fill" else tg.TG_PLAN_AOT
    wl, t, (sep, fus) = _twin_sessions(geom, B, dtype, (1, 700), m, 808 + geom.num_q_heads, T, 48, merge)
    say(f"append in decode {geom} {dtype} {mode} merge={merge}: ctx {wl.ctx_len.tolist()}, {T} steps")
    rng = np.random.default_rng(31)
    for step in range(1, T + 1):
        _step_inputs(rng, sep, dtype)
        for name in ("k_tok", "v_tok", "q"):
            getattr(fus, name).copy_(getattr(sep, name))
        sep.run_decode_step()
        fus.run_decode_step()
        torch.cuda.synchronize()
        assert _same_bits(sep.out, fus.out), f"out differs at step {step}"
        assert _same_bits(sep.lse, fus.lse), f"lse differs at step {step}"
        assert _same_bits(sep.pool, fus.pool), f"pool differs at step {step}"
        assert torch.equal(sep.live_len, fus.live_len), f"live lengths differ at step {step}"
    assert np.array_equal(fus.live_len.cpu().numpy(), t.kv_len + T)
    assert int(sep.full.item()) == 0 and int(fus.full.item()) == 0


def test_append_in_decode_without_room_matches_append_launch():
    """Heads whose table is full take no token in either form: the flag is set, nothing is stored, and the
    attention runs over the full table; the other heads append (matrix-core and generic kernels)."""
    _gpu()
    for geom, dtype in ((Geometry(1, 4, 16, 128, 16, 2), "bf16"), (Geometry(1, 4, 8, 64, 16, 2), "f32")):
        B = 2
        wl = custom(77, geom, B, dtype, [512, 512], budget=np.array([[1.0, 0.5, 0.25, 0.125]]), jitter=0.0)
        t = Tables(wl)
        host = torch.from_numpy(host_pool(wl, t.pool_pages)).to(TORCH_DTYPE[dtype])
        pair = []
        for fused in (False, True):
            s = DecodeSession(wl, tables=t, mode=tg.TG_PLAN_AOT_FILL, n_bins=16, fill="host",
                              pool=host.clone().cuda(), open_end=True)
            s.enable_append(fused=fused)
            pair.append(s)
        sep, fus = pair
        rng = np.random.default_rng(6)
        for step in range(3):
            ks, vs = _step_inputs(rng, sep, dtype)
            for name in ("k_tok", "v_tok", "q"):
                getattr(fus, name).copy_(getattr(sep, name))
            before = _f64(sep.pool)
            live0 = sep.live_len.cpu().numpy()
            sep.run_decode_step()
            fus.run_decode_step()
            torch.cuda.synchronize()
            ref, live, full = oracle.append_token(ks[0], vs[0], before, 0, geom=geom, live_len=live0,
                                                  offsets=t.pt_offsets, pages=t.pt_pages, group_of=t.group_of,
                                                  slot_of=t.slot_of)
            assert sorted(full) == [(0, 0), (0, 2), (1, 0), (1, 2)]
            assert np.array_equal(fus.live_len.cpu().numpy(), live)
            assert np.array_equal(_f64(fus.pool), ref)
            assert _same_bits(sep.out, fus.out) and _same_bits(sep.lse, fus.lse), f"{geom} step {step}"
        assert int(sep.full.item()) == 1 and int(fus.full.item()) == 1


def test_append_in_decode_random_sweep():
    """Seeded sweep: 6 random (dtype, head_dim, KV heads, heads per group, gqa, batch, layers, context range, plan
    mode, bins, merge) cases, each run for a few steps with the append as its own launch and inside the decode
    launch: outputs, lse, the whole pool and the live lengths equal bit for bit after every step."""
    _gpu()
    rng = np.random.default_rng(777)
    for case in range(sweep_cases(6)):
        dtype = ["f32", "bf16"][int(rng.integers(2))]
        d = [64, 128][int(rng.integers(2))]
        H = [1, 2, 4, 8][int(rng.integers(4))]
        hps = [x for x in (1, 2, 4, 8) if H % x == 0]
        Hp = hps[int(rng.integers(len(hps)))]
        gqa = int(rng.integers(1, 17))
        B, L, T = int(rng.integers(1, 5)), int(rng.integers(1, 3)), int(rng.integers(2, 10))
        lo = int(rng.integers(1, 300))
        hi = lo + int(rng.integers(1, 1500))
        mode = [tg.TG_PLAN_AOT_FILL, tg.TG_PLAN_AOT][int(rng.integers(2))]
        n_bins, merge = int(rng.integers(1, 200)), bool(rng.integers(2))
        g = Geometry(L, H, H * gqa, d, 16, Hp)
        say(f"append sweep case {case}: {dtype} d{d} H{H} Hp{Hp} gqa{gqa} B{B} L{L} ctx ({lo}, {hi}) steps {T} "
            f"mode {mode} bins {n_bins} merge {merge}")
        wl, t, (sep, fus) = _twin_sessions(g, B, dtype, (lo, hi), mode, 6000 + case, T, n_bins, merge)
        srng = np.random.default_rng(case)
        for step in range(1, T + 1):
            _step_inputs(srng, sep, dtype)
            for name in ("k_tok", "v_tok", "q"):
                getattr(fus, name).copy_(getattr(sep, name))
            sep.run_decode_step()
            fus.run_decode_step()
            torch.cuda.synchronize()
            assert _same_bits(sep.out, fus.out), f"case {case}: out differs at step {step}"
            assert _same_bits(sep.lse, fus.lse), f"case {case}: lse differs at step {step}"
            assert _same_bits(sep.pool, fus.pool), f"case {case}: pool differs at step {step}"
            assert torch.equal(sep.live_len, fus.live_len), f"case {case}: live lengths differ at step {step}"
        assert int(fus.full.item()) == 0


def test_append_in_noalloc_decode_is_bitwise_append_then_decode():
    """tg_decode_noalloc takes the same append arguments: bitwise equal to tg_append + tg_decode at every step."""
    _gpu()
    g = Geometry(2, 8, 32, 128, 16, 2)
    B, T = 4, 9
    wl, t, (sep, fus) = _twin_sessions(g, B, "bf16", (1, 500), tg.TG_PLAN_AOT_FILL, 919, T, 48, False)
    rng = np.random.default_rng(17)
    for step in range(1, T + 1):
        _step_inputs(rng, sep, "bf16")
        for name in ("k_tok", "v_tok", "q"):
            getattr(fus, name).copy_(getattr(sep, name))
        sep.run_decode_step()
        for l in fus.layers:
            tg.tg_decode_noalloc(fus.append_decode_args[l])
        torch.cuda.synchronize()
        assert _same_bits(sep.out, fus.out) and _same_bits(sep.lse, fus.lse), f"step {step}"
        assert _same_bits(sep.pool, fus.pool) and torch.equal(sep.live_len, fus.live_len), f"step {step}"


@pytest.mark.parametrize("geom,dtype", [(Geometry(1, 4, 16, 128, 16, 2), "bf16"), (Geometry(1, 4, 8, 64, 16, 2), "f32")])
def test_append_in_decode_below_the_open_item_stores_nothing(geom, dtype):
    """A live length below the open item's first entry (lengths that shrank below those the plan was built for)
    is outside the append's contract: the unit takes no token, the flag is set, and its attention is the one
    the same call gives without the append."""
    _gpu()
    B = 3
    wl = custom(55, geom, B, dtype, (300, 900))
    t = Tables(wl, headroom=np.full(B, 8, dtype=np.int32))
    host = torch.from_numpy(host_pool(wl, t.pool_pages)).to(TORCH_DTYPE[dtype])
    pair = []
    for fused in (False, True):
        s = DecodeSession(wl, tables=t, mode=tg.TG_PLAN_AOT_FILL, n_bins=16, fill="host", pool=host.clone().cuda(),
                          open_end=True)
        s.enable_append(fused=fused)
        pair.append(s)
    plain, fus = pair
    rng = np.random.default_rng(8)
    _step_inputs(rng, plain, dtype)
    for name in ("k_tok", "v_tok", "q"):
        getattr(fus, name).copy_(getattr(plain, name))
    # a unit whose open item does not start at entry 0: its live length becomes the item's first entry - 1
    items = fus.plans[0]["items"]
    split_open = [it for it in items if it["tok_end"] < 0 and it["tok_begin"] > 0]
    assert split_open, "the plan has no split unit"
    ub, uh, tb = int(split_open[0]["b"]), int(split_open[0]["kv_head"]), int(split_open[0]["tok_begin"])
    live = plain.live_len.cpu().numpy()
    live[ub, 0, uh] = tb - 1
    plain.live_len.copy_(torch.from_numpy(live).cuda())
    fus.live_len.copy_(torch.from_numpy(live).cuda())
    before = _f64(fus.pool)
    tg.tg_decode(plain.dplans[0].args)       # no append at all
    tg.tg_decode(fus.append_decode_args[0])  # the append: every other unit takes its token
    torch.cuda.synchronize()
    assert int(fus.full.item()) == 1
    got_live = fus.live_len.cpu().numpy()
    expect = live.copy()
    expect[:, 0, :] += 1
    expect[ub, 0, uh] = tb - 1
    assert np.array_equal(got_live, expect)
    # the unit's attention: the same bits as without the append
    G = geom.num_q_heads // geom.num_kv_heads
    a = plain.out[0, ub, uh * G:(uh + 1) * G]
    b = fus.out[0, ub, uh * G:(uh + 1) * G]
    assert _same_bits(a.contiguous(), b.contiguous())
    # nothing was stored for the unit: its reserved rows past its old length are unchanged
    ref, _, full = oracle.append_token(_f64(fus.k_tok[0]), _f64(fus.v_tok[0]), before, 0, geom=geom, live_len=live,
                                       offsets=t.pt_offsets, pages=t.pt_pages, group_of=t.group_of, slot_of=t.slot_of)
    # the oracle appends for the unit at entry tb - 1; the launch must not have: undo that row in the reference
    pg, slot, row = oracle.token_location(ub, 0, uh, tb - 1, num_layers=geom.num_layers, num_groups=geom.num_groups,
                                   page_size=geom.page_size, offsets=t.pt_offsets, pages=t.pt_pages,
                                   group_of=t.group_of, slot_of=t.slot_of)
    ref[pg, :, slot, row] = before[pg, :, slot, row]
    assert np.array_equal(_f64(fus.pool), ref)
