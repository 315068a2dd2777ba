"""Ragged paged decode attention on the GPU (through the C ABI) vs the fp64 oracle.

Small cases compare every output element; the full-size workloads compare
seeded samples of (request, KV head) pairs whose pages are copied back and run
through the oracle one by one.  Unused pool rows are NaN in the small cases so
any read outside a head's retained entries shows up as a non-finite output.
"""
import numpy as np
import pytest
import torch

from gpu_helpers import compare_layer, poisoned_host_pool, sample_pairs, say, sweep_cases
from workloads import Geometry, config, custom

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from paper_2606_06302_amd import tangram as tg
    from paper_2606_06302_amd.runner import DecodeSession, Tables


def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _small_session(wl, mode=0, n_bins=None, split_target=None, free_seed=None, poison=True):
    tables = Tables(wl)
    if free_seed is not None:
        rng = np.random.default_rng(free_seed)
        tables = Tables(wl, free_pages=rng.permutation(tables.pool_pages).astype(np.int32),
                        pool_pages=tables.pool_pages)
    pool = None
    if poison:
        pool = torch.from_numpy(poisoned_host_pool(wl, tables)).to({"f32": torch.float32,
                                                                    "bf16": torch.bfloat16}[wl.dtype]).cuda()
    s = DecodeSession(wl, tables=tables, mode=mode, n_bins=n_bins, split_target=split_target, fill="host",
                      pool=pool)
    s.run_step()
    torch.cuda.synchronize()
    return s


@pytest.mark.parametrize("mode,n_bins,st", [(0, 8, 16), (0, 1, 1), (0, 512, 2048), (0, 3, 40), (1, None, None),
                                            (2, 64, None), (3, 8, None), (3, 300, None)])
def test_config1_tiny_fp32_all_plans(mode, n_bins, st):
    _gpu()
    wl = config(1)
    say(f"config1 mode={mode} n_bins={n_bins} split_target={st}")
    s = _small_session(wl, mode=mode, n_bins=n_bins or 8, split_target=st or 1)
    compare_layer(s, 0, what=f"config1 mode {mode}")


@pytest.mark.parametrize("dtype,d,gqa,Hp,H", [("bf16", 128, 4, 2, 8), ("bf16", 128, 8, 2, 8), ("bf16", 128, 1, 1, 4),
                                              ("bf16", 128, 3, 2, 4), ("bf16", 64, 5, 4, 4), ("bf16", 128, 16, 2, 2),
                                              ("bf16", 128, 5, 4, 4), ("bf16", 128, 7, 1, 2), ("bf16", 128, 12, 2, 2),
                                              ("f32", 128, 2, 2, 4), ("f32", 64, 7, 1, 2), ("bf16", 64, 2, 8, 8)])
def test_shapes_vs_oracle(dtype, d, gqa, Hp, H):
    _gpu()
    g = Geometry(2, H, H * gqa, d, 16, Hp)
    wl = custom(100 + d + gqa * 3 + Hp, g, 3, dtype, (40, 700), kv_scale=0.5)
    say(f"shape dtype={dtype} d={d} gqa={gqa} Hp={Hp} H={H} ctx={wl.ctx_len.tolist()}")
    s = _small_session(wl, n_bins=37, split_target=50)
    for l in range(2):
        compare_layer(s, l, what=f"{dtype} d{d} gqa{gqa} layer {l}")


def test_config2_shape_scaled_plan_modes_agree():
    _gpu()
    g = Geometry(1, 8, 32, 128, 16, 2)
    wl = custom(2002, g, 6, "bf16", 2048, kv_scale=0.5)
    outs = []
    for mode, nb, stg in [(0, 512, 2048), (0, 7, 9), (1, 1, 1), (2, 100, 1), (3, 512, 1), (3, 5, 1)]:
        say(f"config2-scaled mode={mode} n_bins={nb}")
        s = _small_session(wl, mode=mode, n_bins=nb, split_target=stg)
        compare_layer(s, 0, what=f"mode {mode}")
        outs.append(s.out.float().cpu())
    for o in outs[1:]:
        assert torch.allclose(o, outs[0], atol=2e-2, rtol=0)


def test_single_retained_token_returns_value_exactly():
    _gpu()
    g = Geometry(1, 4, 8, 128, 16, 2)
    wl = custom(77, g, 3, "bf16", (100, 900), budget=np.full((1, 4), 1e-6), jitter=0.0)
    s = _small_session(wl, n_bins=5, split_target=5)
    t = s.t
    assert np.all(t.kv_len == 1)
    out = s.out[0].cpu()
    for b in range(wl.batch):
        for h in range(4):
            page = int(t.pt_pages[t.pt_offsets[b * 2 + t.group_of[0, h]]])
            v = s.pool[page, 1, int(t.slot_of[0, h]), 0].cpu()
            for j in range(2):
                assert torch.equal(out[b, h * 2 + j], v), (b, h, j)


def test_page_placement_invariance_is_bitwise():
    _gpu()
    g = Geometry(1, 8, 32, 128, 16, 2)
    wl = custom(303, g, 4, "bf16", (500, 3000), kv_scale=0.5)
    t1 = Tables(wl)
    # same logical contents at a different physical placement
    rng = np.random.default_rng(5)
    free2 = rng.permutation(t1.pool_pages).astype(np.int32)
    t2 = Tables(wl, free_pages=free2, pool_pages=t1.pool_pages)
    pool1 = torch.from_numpy(poisoned_host_pool(wl, t1)).to(torch.bfloat16).cuda()
    pool2 = torch.full_like(pool1, float("nan"))
    pool2[torch.from_numpy(t2.pt_pages.astype(np.int64)).cuda()] = pool1[torch.from_numpy(t1.pt_pages.astype(np.int64)).cuda()]
    s1 = DecodeSession(wl, tables=t1, n_bins=40, split_target=90, fill="host", pool=pool1)
    s2 = DecodeSession(wl, tables=t2, n_bins=40, split_target=90, fill="host", pool=pool2)
    s1.run_step()
    s2.run_step()
    torch.cuda.synchronize()
    assert torch.equal(s1.out, s2.out)
    compare_layer(s1, 0, what="placement")


def test_empty_bins_and_single_bin():
    _gpu()
    g = Geometry(1, 2, 4, 128, 16, 1)
    wl = custom(9, g, 1, "bf16", 300)
    for nb, stg in [(1, 1), (300, 1), (300, 1000)]:
        say(f"bins={nb} split_target={stg}")
        s = _small_session(wl, n_bins=nb, split_target=stg)
        compare_layer(s, 0, what=f"bins {nb}")


def test_negative_controls_fail():
    """Corrupting the page table or a length must break parity (the check is not vacuous)."""
    _gpu()
    g = Geometry(1, 8, 32, 128, 16, 2)
    wl = custom(404, g, 4, "bf16", 4096, kv_scale=0.5, budget=np.full((1, 8), 0.5), jitter=0.0)
    s = _small_session(wl, n_bins=64, split_target=64, poison=False)
    compare_layer(s, 0, what="baseline")
    # point request 0's first page at the last request's last page (a page of
    # another table; swapping pages inside one table would only permute tokens)
    good = s.t.d_pt_pages.clone()
    bad = good.clone()
    bad[[0, -1]] = good[[-1, 0]]
    s.t.d_pt_pages.copy_(bad)
    s.run_step()
    torch.cuda.synchronize()
    with pytest.raises(AssertionError):
        compare_layer(s, 0, pairs=[(0, h) for h in range(8)], check_lse=False, what="swapped pages")
    s.t.d_pt_pages.copy_(good)
    # drop the last page of one head: plan from a shortened length
    kv = s.t.kv_len.copy()
    kv[1, 0, 3] -= 16
    plan = tg.tg_build_plan(g, 4, 0, kv, s.t.pt_offsets, s.t.group_of, s.t.slot_of, 0, 64, 64)
    from paper_2606_06302_amd.device import bind_decode, upload_plan
    dp = upload_plan(g, 4, plan, "cuda")
    bind_decode(dp, g, 4, tg.TG_BF16, s.q[0], s.pool, s.t.d_pt_pages, s.out[0], s.lse[0])
    tg.tg_decode(dp.args)
    torch.cuda.synchronize()
    with pytest.raises(AssertionError):
        compare_layer(s, 0, pairs=[(1, 3)], check_lse=False, what="short head")


@pytest.mark.parametrize("cfg", [2, 4])
def test_full_size_config_sampled(cfg):
    _gpu()
    wl = config(cfg)
    say(f"config {cfg} full size: B={wl.batch} ctx range {wl.ctx_len.min()}..{wl.ctx_len.max()}")
    for mode in (0, 1, 3):
        s = DecodeSession(wl, mode=mode)
        s.run_step()
        torch.cuda.synchronize()
        pairs = sample_pairs(wl, 24, seed=cfg)
        if cfg == 4:   # always include the longest unit
            b = int(np.argmax(wl.ctx_len))
            h = int(np.argmax(s.t.kv_len[b, 0]))
            pairs = sorted(set(pairs) | {(b, h)})
        compare_layer(s, 0, pairs=pairs, what=f"config {cfg} mode {mode}")
        del s
        torch.cuda.empty_cache()


@pytest.mark.parametrize("plan", ["aot", "fill-graph"])
def test_full_size_config3_sampled(plan):
    """Config 3 at full size (64 layers, batch 64).  "fill-graph" is exactly what bench.py times: the
    sequential-fill plan (TG_PLAN_AOT_FILL) on tg_decode_max_ctas bins, the 64 layers' launches captured in a
    HIP graph; the replays must equal the eager step bit for bit, and sampled (request, KV head) pairs of
    sampled layers match the oracle.  "aot" is the LPT-binned proportional plan, run eagerly."""
    _gpu()
    wl = config(3)
    mode = tg.TG_PLAN_AOT if plan == "aot" else tg.TG_PLAN_AOT_FILL
    n_cta = tg.tg_decode_max_ctas(wl.geom, tg.TG_BF16, 0)
    say(f"config 3 full size: 64 layers, B=64, plan {plan}, {n_cta} bins")
    s = DecodeSession(wl, mode=mode)
    assert s.n_bins == n_cta
    s.run_step()
    torch.cuda.synchronize()
    if plan == "fill-graph":
        eager_out, eager_lse = s.out.clone(), s.lse.clone()
        st = torch.cuda.Stream()
        graph = s.capture_step(st)
        for rep in range(2):
            s.out.zero_()
            s.lse.zero_()
            torch.cuda.synchronize()
            graph.replay()
            torch.cuda.synchronize()
            assert torch.equal(s.out, eager_out) and torch.equal(s.lse, eager_lse), rep
        del eager_out, eager_lse
    rng = np.random.default_rng(33)
    for layer in sorted(rng.choice(64, size=4, replace=False).tolist()):
        compare_layer(s, layer, pairs=sample_pairs(wl, 10, seed=layer), what=f"config 3 {plan} layer {layer}")
    del s
    torch.cuda.empty_cache()


@pytest.mark.parametrize("dtype,d,gqa", [("bf16", 128, 8), ("f32", 64, 2)])
def test_worker_timestamps(dtype, d, gqa):
    """The optional per-worker stamps: ordered, present for every bin (empty bins
    stamp start == end), and the outputs stay bitwise identical."""
    _gpu()
    from paper_2606_06302_amd import tangram as tg
    g = Geometry(1, 4, 4 * gqa, d, 16, 2)
    wl = custom(880 + d, g, 3, dtype, (40, 2000), kv_scale=0.5)
    s = _small_session(wl, mode=0, n_bins=50, split_target=60)
    ref = s.out.clone()
    dp = s.dplans[0]
    nb = dp.host["num_bins"]
    ts = torch.full((2 * nb,), -1, dtype=torch.int64, device="cuda")
    args = tg.tg_decode_args.from_buffer_copy(dp.args)
    args.timestamps = ts.data_ptr()
    s.out.zero_()
    tg.tg_decode(args)
    torch.cuda.synchronize()
    assert torch.equal(s.out, ref)
    t = ts.view(-1, 2).cpu().numpy()
    assert (t >= 0).all() and (t[:, 1] >= t[:, 0]).all()
    empty = np.diff(s.plans[0]["bin_offsets"]) == 0
    assert (t[empty, 1] == t[empty, 0]).all()
    busy = s.worker_busy()
    assert len(busy) == 1 and busy[0][0] >= busy[0][1] > 0


def test_graph_replay_matches_eager_bitwise():
    """A captured step replayed several times, with eager work and synchronisation
    in between, reproduces the eager outputs bit for bit on every replay."""
    _gpu()
    g = Geometry(3, 8, 64, 128, 16, 2)
    wl = custom(1357, g, 4, "bf16", (200, 4000), kv_scale=0.5)
    s = _small_session(wl, mode=3, n_bins=64)
    ref_out, ref_lse = s.out.clone(), s.lse.clone()
    st = torch.cuda.Stream()
    graph = s.capture_step(st)
    for rep in range(4):
        s.out.zero_()
        s.lse.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(s.out, ref_out), rep
        assert torch.equal(s.lse, ref_lse), rep
        s.run_step()          # eager work between replays
        torch.cuda.synchronize()
        assert torch.equal(s.out, ref_out), rep


@pytest.mark.parametrize("per_layer", [False, True])
def test_xcd_calibrated_fill_plan_matches_oracle(per_layer):
    """The per-XCD calibration rebuilds the fill plan with bin weights (one set, or
    one per layer as the benchmark uses); the new plan still computes the same
    attention (oracle) as the unweighted one."""
    _gpu()
    g = Geometry(2, 8, 64, 128, 16, 2)
    wl = custom(2468, g, 6, "bf16", (300, 5000), kv_scale=0.5)
    s = _small_session(wl, mode=3, n_bins=128)
    ref = s.out.clone()
    speed = s.calibrate_xcd_weights(per_layer=per_layer)
    assert speed.shape == ((2, 8) if per_layer else (8,)) and np.all(speed > 0) and s.bin_weights is not None
    s.run_step()
    torch.cuda.synchronize()
    for l in range(2):
        compare_layer(s, l, what=f"calibrated layer {l}")
    assert torch.allclose(s.out.float(), ref.float(), atol=2e-2, rtol=0)


def test_split_map_plan_vs_oracle():
    """Algorithm 1's split map executed as is (S[l][g] workers per head group) gives the same attention."""
    _gpu()
    g = Geometry(2, 8, 32, 128, 16, 2)
    wl = custom(321, g, 6, "bf16", (100, 4000))
    say(f"split-map plan: ctx {wl.ctx_len.tolist()}")
    s = DecodeSession(wl, mode=tg.TG_PLAN_SPLIT_MAP, n_bins=128, fill="host")
    s.run_step()
    torch.cuda.synchronize()
    for l in range(g.num_layers):
        assert s.plans[l]["num_bins"] == int(tg.tg_split_map(g, wl.budget, s.t.perm, 128)[l].sum())
        compare_layer(s, l, what=f"split map layer {l}")


@pytest.mark.parametrize("gqa,mode,n_bins,st", [(8, 3, 64, 1), (8, 0, 512, 4096), (16, 0, 300, 900), (3, 3, 97, 1),
                                                (1, 4, 128, 1), (8, 3, 1, 1), (5, 0, 2000, 8000)])
def test_fused_merge_matches_two_launch_merge_bitwise(gqa, mode, n_bins, st):
    """The in-launch merge (each split piece counts itself on its unit's counter; the piece that arrives last
    merges) gives bit for bit the outputs and LSEs of the separate merge launch, including plans that cut units
    into dozens of pieces, on repeated calls (the counters are back at zero after each); both match the oracle."""
    _gpu()
    g = Geometry(2, 8, 8 * gqa, 128, 16, 2)
    wl = custom(7300 + gqa + n_bins, g, 5, "bf16", (100, 8000), kv_scale=0.5)
    tables = Tables(wl)
    pool = torch.from_numpy(poisoned_host_pool(wl, tables)).to(torch.bfloat16).cuda()
    kw = dict(tables=tables, mode=mode, n_bins=n_bins, split_target=st, fill="host", pool=pool)
    if mode == tg.TG_PLAN_SPLIT_MAP:
        kw["n_bins"] = n_bins
    fused = DecodeSession(wl, fused_merge=True, **kw)
    assert fused.merge_counters is not None
    twol = DecodeSession(wl, fused_merge=False, q=fused.q, **kw)
    splits = [int(fused.plans[l]["unit_splits"].max()) for l in fused.layers]
    say(f"fused merge gqa {gqa} mode {mode} bins {n_bins}: partials "
        f"{[fused.plans[l]['num_partials'] for l in fused.layers]}, most splits per unit {splits}")
    twol.run_step()
    for rep in range(3):
        fused.out.fill_(float("nan"))
        fused.lse.fill_(float("nan"))
        fused.run_step()
        torch.cuda.synchronize()
        assert torch.equal(fused.out, twol.out) and torch.equal(fused.lse, twol.lse), rep
        assert int(fused.merge_counters.abs().sum().item()) == 0
    for l in fused.layers:
        compare_layer(fused, l, what=f"fused merge layer {l}")


def test_read_probe_checksums():
    """The streaming-read probe reads exactly the slabs the decode reads: every worker's XOR checksum equals
    the host's over the same (page, slot) K and V slabs."""
    _gpu()
    wl = config(1)
    s = DecodeSession(wl, n_bins=8, split_target=16, fill="host")
    pages, slots = s.layer_slabs(0)
    pool = s.pool.contiguous()
    n_workers = 7
    out = torch.zeros(n_workers, dtype=torch.int32, device="cuda")
    tg.tg_read_probe(wl.geom, tg.TG_F32, pool, torch.from_numpy(pages).cuda(), torch.from_numpy(slots).cuda(),
                     n_workers, out)
    torch.cuda.synchronize()
    words = pool.cpu().numpy().view(np.uint32).reshape(s.t.pool_pages, 2, wl.geom.heads_per_group, -1)
    n = len(pages)
    want = []
    for w in range(n_workers):
        lo, hi = n * w // n_workers, n * (w + 1) // n_workers
        x = np.uint32(0)
        for i in range(lo, hi):
            x ^= np.bitwise_xor.reduce(words[pages[i], 0, slots[i]]) ^ np.bitwise_xor.reduce(words[pages[i], 1, slots[i]])
        want.append(int(x))
    assert out.cpu().numpy().view(np.uint32).tolist() == want
    assert n == int(sum(-(-(it["tok_end"] - it["tok_begin"]) // 16) for it in s.plans[0]["items"]))


def test_random_shapes_and_plans_sweep():
    """Seeded sweep: 16 random (dtype, head_dim, KV heads, heads per group, gqa, batch, layers, context range,
    plan mode, bins, split target) cases, every layer against the oracle, pool rows past the retained
    lengths poisoned with NaN."""
    _gpu()
    rng = np.random.default_rng(4242)
    for case in range(sweep_cases(16)):
        dtype = ["f32", "bf16"][int(rng.integers(2))]
        d = [64, 128][int(rng.integers(2))]
        H = [1, 2, 4, 8][int(rng.integers(4))]
        Hp = [x for x in (1, 2, 4, 8) if H % x == 0][int(rng.integers(len([x for x in (1, 2, 4, 8) if H % x == 0])))]
        gqa = int(rng.integers(1, 17))
        B, L = int(rng.integers(1, 5)), int(rng.integers(1, 3))
        lo = int(rng.integers(1, 400))
        hi = lo + int(rng.integers(0, 2500))
        mode = int(rng.integers(0, 4))
        n_bins, st = int(rng.integers(1, 300)), int(rng.integers(1, 500))
        g = Geometry(L, H, H * gqa, d, 16, Hp)
        wl = custom(5000 + case, g, B, dtype, (lo, hi) if hi > lo else lo, kv_scale=0.5)
        say(f"sweep case {case}: {dtype} d{d} H{H} Hp{Hp} gqa{gqa} B{B} L{L} ctx={wl.ctx_len.tolist()} "
            f"mode {mode} bins {n_bins} split {st}")
        s = _small_session(wl, mode=mode, n_bins=n_bins, split_target=st)
        for l in range(L):
            compare_layer(s, l, what=f"sweep case {case} layer {l}")
