"""Pins of the fp64 oracle against facts fixed outside the oracle itself.

Each test checks one oracle function against something it cannot simply echo:
hand-derived values for the tiny workload (tests/golden/config1_hand.json),
brute force over tiny inputs, closed forms, library routines that compute the
same quantity by another road (torch's scaled_dot_product_attention), and
invariants of the method (placement and split invariance, Graham's bound).
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
from workloads import Geometry

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "config1_hand.json")))


def cfg1_arrays():
    budget = np.array(GOLD["budget"], dtype=np.float64)
    ratio = np.broadcast_to(budget, (2, 1, 4)).copy()
    ctx = np.array(GOLD["ctx_len"])
    return budget, ratio, ctx


# ---------------------------------------------------------------- Eq. 4

def test_lengths_config1_hand():
    _, ratio, ctx = cfg1_arrays()
    assert oracle.retained_lengths(ratio, ctx).tolist() == GOLD["kv_len"]


def test_lengths_fp64_product_then_ceil():
    # 0.07*100 evaluates to 7.000000000000001 in fp64, 0.29*100 to 28.999999999999996.
    assert oracle.retained_lengths(np.array([[[0.07]]]), [100])[0, 0, 0] == 8
    assert oracle.retained_lengths(np.array([[[0.29]]]), [100])[0, 0, 0] == 29
    assert oracle.retained_lengths(np.array([[[1.0]]]), [65536])[0, 0, 0] == 65536
    assert oracle.retained_lengths(np.array([[[1e-9]]]), [131072])[0, 0, 0] == 1


def test_lengths_bruteforce_scan():
    rng = np.random.default_rng(7)
    for _ in range(300):
        n = int(rng.integers(1, 400))
        r = float(rng.choice([rng.uniform(1e-4, 1.0), rng.integers(1, 64) / 64.0]))
        got = int(oracle.retained_lengths(np.array([[[r]]]), [n])[0, 0, 0])
        prod = np.float64(r) * np.float64(n)
        k = 0
        while k < prod:          # smallest integer not below the fp64 product
            k += 1
        assert got == k and 1 <= got <= n


@pytest.mark.parametrize("bad", [0.0, -0.1, 1.0000001, float("nan"), float("inf")])
def test_lengths_reject_bad_ratio(bad):
    with pytest.raises(oracle.OracleError):
        oracle.retained_lengths(np.array([[[bad]]]), [10])


# ------------------------------------------------------- clustering (4.2.2)

def test_cluster_config1_hand():
    budget, _, _ = cfg1_arrays()
    perm, group_of, slot_of = oracle.cluster_heads(budget, 2)
    assert perm.tolist() == GOLD["perm"]
    assert group_of.tolist() == GOLD["group_of"]
    assert slot_of.tolist() == GOLD["slot_of"]


def test_cluster_ties_are_stable_and_adjacent_is_identity():
    perm, _, _ = oracle.cluster_heads(np.array([[0.5, 0.2, 0.5, 0.2]]), 2)
    assert perm.tolist() == [[1, 3, 0, 2]]
    perm, g, s = oracle.cluster_heads(np.array([[0.9, 0.1, 0.5, 0.2]]), 2, oracle.GROUP_ADJACENT)
    assert perm.tolist() == [[0, 1, 2, 3]] and g.tolist() == [[0, 0, 1, 1]] and s.tolist() == [[0, 1, 0, 1]]


def _equal_partitions(items, k):
    """All partitions of `items` into blocks of size k (brute force)."""
    if not items:
        yield []
        return
    first, rest = items[0], items[1:]
    for others in itertools.combinations(rest, k - 1):
        remaining = [x for x in rest if x not in others]
        for tail in _equal_partitions(remaining, k):
            yield [(first,) + others] + tail


@pytest.mark.parametrize("H,Hp", [(4, 2), (6, 2), (6, 3), (8, 2), (8, 4)])
def test_cluster_minimises_sum_of_group_maxima(H, Hp):
    """Sorting then cutting minimises the pages held by group maxima (the
    exchange argument behind Budget-Aware Clustering), checked by brute force."""
    rng = np.random.default_rng(H * 10 + Hp)
    for _ in range(20):
        b = rng.uniform(0.01, 1.0, size=H)
        _, group_of, _ = oracle.cluster_heads(b[None, :], Hp)
        clustered = sum(max(b[h] for h in range(H) if group_of[0, h] == g) for g in range(H // Hp))
        best = min(sum(max(b[list(blk)]) for blk in part) for part in _equal_partitions(list(range(H)), Hp))
        assert clustered == pytest.approx(best, abs=1e-15)


def test_cluster_rejects_indivisible_groups():
    with pytest.raises(oracle.OracleError):
        oracle.cluster_heads(np.full((1, 6), 0.5), 4)


# --------------------------------------------------- reservation (4.1, 4.2.1)

def test_reserve_config1_hand():
    budget, ratio, ctx = cfg1_arrays()
    _, group_of, _ = oracle.cluster_heads(budget, 2)
    res = oracle.reserve(ratio, ctx, group_of, 2, 16, np.arange(100))
    assert res["group_len"].tolist() == GOLD["group_len"]
    assert res["offsets"].tolist() == GOLD["offsets"]
    assert res["pages_needed"] == GOLD["pages_needed"]
    assert res["pages"].tolist() == list(range(80))
    perm_free = np.random.default_rng(3).permutation(100)
    res2 = oracle.reserve(ratio, ctx, group_of, 2, 16, perm_free)
    assert res2["pages"].tolist() == perm_free[:80].tolist()


def test_reserve_invariants_random():
    rng = np.random.default_rng(11)
    for trial in range(40):
        H = int(rng.choice([2, 4, 6, 8]))
        Hp = int(rng.choice([d for d in (1, 2, 3, 4, 8) if H % d == 0]))
        L, Bn, P = int(rng.integers(1, 4)), int(rng.integers(1, 5)), int(rng.choice([1, 4, 16]))
        budget = rng.uniform(0.01, 1.0, size=(L, H))
        ratio = np.clip(budget[None] + rng.uniform(-0.03, 0.03, size=(Bn, L, H)), 0.02, 1.0)
        ctx = rng.integers(1, 300, size=Bn)
        _, group_of, _ = oracle.cluster_heads(budget, Hp)
        G = H // Hp
        free = rng.permutation(20000)
        res = oracle.reserve(ratio, ctx, group_of, G, P, free)
        off, pages = res["offsets"], res["pages"]
        assert np.all(np.diff(off) >= 0) and off[0] == 0 and off[-1] == len(pages)
        assert len(set(pages.tolist())) == len(pages) and set(pages.tolist()) <= set(free.tolist())
        for b in range(Bn):
            for l in range(L):
                for g in range(G):
                    cap = (off[(b * L + l) * G + g + 1] - off[(b * L + l) * G + g]) * P
                    members = [res["kv_len"][b, l, h] for h in range(H) if group_of[l, h] == g]
                    assert max(members) <= cap < max(members) + P
        # too short a free list: error, nothing consumed
        short = free[: res["pages_needed"] - 1].copy()
        before = short.copy()
        with pytest.raises(oracle.OutOfPages):
            oracle.reserve(ratio, ctx, group_of, G, P, short)
        assert np.array_equal(short, before)


# ----------------------------------------------------------- Algorithm 1

def test_split_map_config1_hand():
    budget, _, _ = cfg1_arrays()
    perm2, _, _ = oracle.cluster_heads(budget, 2)
    perm1, _, _ = oracle.cluster_heads(budget, 1)
    assert oracle.split_map(budget, perm2, 2, 256).tolist() == GOLD["split_map"]["hp2_ncta256"]
    assert oracle.split_map(budget, perm2, 2, 8).tolist() == GOLD["split_map"]["hp2_ncta8"]
    assert oracle.split_map(budget, perm1, 1, 256).tolist() == GOLD["split_map"]["hp1_ncta256"]


def test_split_map_round_half_up_and_floor_of_one():
    b = np.array([[0.5, 0.5, 0.5, 0.5]])
    perm, _, _ = oracle.cluster_heads(b, 1)
    assert oracle.split_map(b, perm, 1, 10).tolist() == [[3, 3, 3, 3]]     # 2.5 rounds up
    b = np.array([[0.25, 0.75]])
    perm, _, _ = oracle.cluster_heads(b, 1)
    assert oracle.split_map(b, perm, 1, 2).tolist() == [[1, 2]]            # 0.5 -> 1, 1.5 -> 2
    b = np.array([[0.001, 1.0]])
    perm, _, _ = oracle.cluster_heads(b, 1)
    assert oracle.split_map(b, perm, 1, 4).tolist() == [[1, 4]]            # max(1, 0) = 1


def test_split_map_proportional():
    rng = np.random.default_rng(5)
    for _ in range(50):
        L, H, Hp, n = 3, 8, int(rng.choice([1, 2, 4])), int(rng.integers(8, 1024))
        b = rng.uniform(0.02, 1.0, size=(L, H))
        perm, _, _ = oracle.cluster_heads(b, Hp)
        S = oracle.split_map(b, perm, Hp, n)
        for l in range(L):
            for i in range(H // Hp):
                exact = sum(b[l, perm[l, j]] for j in range(i * Hp, (i + 1) * Hp)) * n / b[l].sum()
                assert abs(S[l, i] - max(exact, 1.0)) <= 0.5 + 1e-9 or (exact < 0.5 and S[l, i] == 1)


# ------------------------------------------------------------ partition

def _cfg1_plan(mode=oracle.MODE_AOT, n_bins=8, split_target=16, free=None, bin_weights=None):
    budget, ratio, ctx = cfg1_arrays()
    _, group_of, slot_of = oracle.cluster_heads(budget, 2)
    res = oracle.reserve(ratio, ctx, group_of, 2, 16, np.arange(100) if free is None else free)
    plan = oracle.partition_plan(res["kv_len"], res["offsets"], group_of, slot_of, 0, num_layers=1,
                                 num_groups=2, page_size=16, mode=mode, n_bins=n_bins,
                                 split_target=split_target, bin_weights=bin_weights)
    return res, group_of, slot_of, plan


def _random_case(rng):
    H, Hp, L, Bn, P = 8, int(rng.choice([1, 2, 4])), 2, int(rng.integers(1, 6)), int(rng.choice([1, 4, 16]))
    budget = rng.uniform(0.01, 1.0, size=(L, H))
    ratio = np.clip(budget[None] + rng.uniform(-.03, .03, size=(Bn, L, H)), 0.02, 1.0)
    ctx = rng.integers(1, 700, size=Bn)
    _, group_of, slot_of = oracle.cluster_heads(budget, Hp)
    G = H // Hp
    res = oracle.reserve(ratio, ctx, group_of, G, P, np.arange(100000))
    return dict(res=res, L=L, G=G, P=P, group_of=group_of, slot_of=slot_of)


def test_plan_config1_hand():
    _, _, _, plan = _cfg1_plan()
    gold = GOLD["plan_split_target16_bins8"]
    assert plan["unit_splits"].tolist() == gold["unit_splits"]
    assert plan["unit_partial_base"].tolist() == gold["unit_partial_base"]
    assert plan["num_partials"] == gold["num_partials"]
    assert plan["bin_load"].tolist() == gold["bin_load"]
    assert plan["bin_offsets"].tolist() == gold["bin_offsets"]
    assert [list(it) for it in plan["items"]] == gold["items"]
    assert max(gold["bin_load"]) / np.mean(gold["bin_load"]) == pytest.approx(256 / 240)


def test_fill_plan_config1_hand():
    _, _, _, plan = _cfg1_plan(mode=oracle.MODE_FILL, n_bins=8)
    gold = GOLD["plan_fill_bins8"]
    assert [list(it) for it in plan["items"]] == gold["items"]
    assert plan["bin_offsets"].tolist() == gold["bin_offsets"]
    assert plan["bin_load"].tolist() == gold["bin_load"]
    assert plan["unit_splits"].tolist() == gold["unit_splits"] and plan["num_partials"] == gold["num_partials"]


def uniform_gold_items(gold):
    """The hand-derived UNIFORM plan's items, spelled out from its per-head chunk bounds."""
    items = []
    for b in range(2):
        for h in range(4):
            bounds = gold["chunk_bounds"][f"head{h}"]
            pt_base, slot = gold["table_and_slot"][b][h]
            base = gold["unit_partial_base"][b][h]
            for c in range(len(bounds) - 1):
                items.append([pt_base, b, h, slot, bounds[c], bounds[c + 1], base + c])
    return items


def test_uniform_plan_config1_hand():
    """Static uniform splits (the straggler baseline): 8 splits per unit capped by its pages, one bin per
    chunk; a floor-for-ceil slip in the split count or a chunk-boundary slip changes these values."""
    gold = GOLD["plan_uniform_bins64"]
    _, _, _, plan = _cfg1_plan(mode=oracle.MODE_UNIFORM, n_bins=gold["n_bins"])
    assert plan["unit_splits"].tolist() == gold["unit_splits"]
    assert plan["unit_partial_base"].tolist() == gold["unit_partial_base"]
    assert plan["num_partials"] == gold["num_partials"] == 56
    assert plan["bin_offsets"].tolist() == list(range(gold["num_bins"] + 1))
    assert plan["bin_load"].tolist() == gold["bin_load"]
    assert [list(it) for it in plan["items"]] == uniform_gold_items(gold)
    # n_bins just above a multiple of the unit count: the ceiling gives one more split per unit
    _, _, _, plan9 = _cfg1_plan(mode=oracle.MODE_UNIFORM, n_bins=57)
    assert plan9["unit_splits"].tolist() == [[8, 8, 8, 4], [8, 8, 8, 4]]
    _, _, _, plan7 = _cfg1_plan(mode=oracle.MODE_UNIFORM, n_bins=9)
    assert plan7["unit_splits"].tolist() == [[2, 2, 2, 2], [2, 2, 2, 2]]


def test_naive_plan_config1_hand():
    gold = GOLD["plan_naive"]
    for n_bins in (1, 8, 64):          # the bin count is not an input of the naive split
        _, _, _, plan = _cfg1_plan(mode=oracle.MODE_NAIVE, n_bins=n_bins)
        assert [list(it) for it in plan["items"]] == gold["items"]
        assert plan["bin_offsets"].tolist() == gold["bin_offsets"]
        assert plan["unit_splits"].tolist() == gold["unit_splits"]
        assert plan["unit_partial_base"].tolist() == gold["unit_partial_base"]
        assert plan["num_partials"] == gold["num_partials"] == 0
        assert plan["bin_load"].tolist() == gold["bin_load"]


def test_plan_reduces_to_algorithm1():
    """One request, P=1 and lengths exactly B*N: the executed split counts are
    Algorithm 1's split map with H_p = 1."""
    budget = np.array([[1.0, 0.5, 0.25, 0.125]])
    kv = np.array([[[4096, 2048, 1024, 512]]])
    perm, group_of, slot_of = oracle.cluster_heads(budget, 1)
    offsets = np.concatenate([[0], np.cumsum(kv[0, 0][np.argsort(group_of[0])])])
    plan = oracle.partition_plan(kv, offsets, group_of, slot_of, 0, num_layers=1, num_groups=4,
                                 page_size=1, mode=oracle.MODE_AOT, n_bins=16, split_target=256)
    S = oracle.split_map(budget, perm, 1, 256)
    assert [int(plan["unit_splits"][0, perm[0, i]]) for i in range(4)] == S[0].tolist() == [17, 34, 68, 137]


def _check_plan_invariants(plan, kv, offsets, group_of, slot_of, layer, L, G, P, n_bins, mode):
    Bn, _, H = kv.shape
    items = plan["items"]
    bo = plan["bin_offsets"]
    assert bo[0] == 0 and bo[-1] == len(items) and np.all(np.diff(bo) >= 0)
    if mode == oracle.MODE_AOT:
        assert len(bo) == n_bins + 1
        loads = plan["bin_load"]
        assert loads.max() <= loads.mean() + max(it[5] - it[4] for it in items) + 1e-9   # Graham's LPT bound
    if mode == oracle.MODE_FILL:
        assert len(bo) == n_bins + 1
        # every bin holds floor or ceil of total/n_bins pages
        pages = [sum(-(-(it[5] - it[4] + it[4] % P) // P) for it in items[bo[k]:bo[k + 1]]) for k in range(n_bins)]
        total = sum(-(-kv[b, layer, h] // P) for b in range(kv.shape[0]) for h in range(kv.shape[2]))
        assert sum(pages) == total and max(pages) - min(pages) <= 1
    seen = {}
    for (pt_base, b, h, slot, t0, t1, out_idx) in items:
        assert pt_base == offsets[(b * L + layer) * G + group_of[layer, h]] and slot == slot_of[layer, h]
        assert t0 % P == 0 and 0 <= t0 < t1 <= kv[b, layer, h]
        seen.setdefault((b, h), []).append((t0, t1, out_idx))
    nparts = 0
    for b in range(Bn):
        for h in range(H):
            ch = sorted(seen[(b, h)])
            assert ch[0][0] == 0 and ch[-1][1] == kv[b, layer, h]
            assert all(ch[i][1] == ch[i + 1][0] for i in range(len(ch) - 1))
            s = plan["unit_splits"][b, h]
            assert len(ch) == s
            if s == 1:
                assert ch[0][2] == -1 and plan["unit_partial_base"][b, h] == -1
            else:
                base = plan["unit_partial_base"][b, h]
                assert sorted(c[2] for c in ch) == list(range(base, base + s))
                nparts += s
    assert nparts == plan["num_partials"]


@pytest.mark.parametrize("mode", [oracle.MODE_AOT, oracle.MODE_NAIVE, oracle.MODE_UNIFORM, oracle.MODE_FILL])
def test_plan_invariants_random(mode):
    rng = np.random.default_rng(21 + mode)
    for _ in range(25):
        H, Hp, L, Bn, P = 8, int(rng.choice([1, 2, 4])), 2, int(rng.integers(1, 6)), int(rng.choice([1, 4, 16]))
        budget = rng.uniform(0.01, 1.0, size=(L, H))
        ratio = np.clip(budget[None] + rng.uniform(-.03, .03, size=(Bn, L, H)), 0.02, 1.0)
        ctx = rng.integers(1, 700, size=Bn)
        _, group_of, slot_of = oracle.cluster_heads(budget, Hp)
        G = H // Hp
        res = oracle.reserve(ratio, ctx, group_of, G, P, np.arange(100000))
        n_bins, st = int(rng.integers(1, 40)), int(rng.integers(1, 200))
        layer = int(rng.integers(0, L))
        plan = oracle.partition_plan(res["kv_len"], res["offsets"], group_of, slot_of, layer, num_layers=L,
                                     num_groups=G, page_size=P, mode=mode, n_bins=n_bins, split_target=st)
        _check_plan_invariants(plan, res["kv_len"], res["offsets"], group_of, slot_of, layer, L, G, P, n_bins, mode)
        again = oracle.partition_plan(res["kv_len"], res["offsets"], group_of, slot_of, layer, num_layers=L,
                                      num_groups=G, page_size=P, mode=mode, n_bins=n_bins, split_target=st)
        assert again["items"] == plan["items"]


# ------------------------------------------------------------ attention

def write_dense(pool, dense_k, dense_v, kv_len, offsets, pages, group_of, slot_of, L, G, P):
    """Scatter dense per-head rows into the paged pool, page layout
    [page][K|V][slot][row][d] (test-side writer, independent of the oracle's reader)."""
    Bn, _, H = kv_len.shape
    for b in range(Bn):
        for l in range(L):
            for h in range(H):
                base = offsets[(b * L + l) * G + group_of[l, h]]
                for i in range(kv_len[b, l, h]):
                    page = pages[base + i // P]
                    pool[page, 0, slot_of[l, h], i % P] = dense_k[b, l, h, i]
                    pool[page, 1, slot_of[l, h], i % P] = dense_v[b, l, h, i]


def small_case(seed, Bn=2, L=2, H=4, gqa=2, d=8, Hp=2, P=4, ctx=(5, 40), ratio=None, free_seed=None):
    rng = np.random.default_rng(seed)
    g = Geometry(L, H, H * gqa, d, P, Hp)
    budget = rng.uniform(0.05, 1.0, size=(L, H))
    if ratio is None:
        ratio = np.clip(budget[None] + rng.uniform(-.03, .03, size=(Bn, L, H)), 0.02, 1.0)
    ctxv = rng.integers(ctx[0], ctx[1] + 1, size=Bn)
    _, group_of, slot_of = oracle.cluster_heads(budget, Hp)
    res = oracle.reserve(ratio, ctxv, group_of, H // Hp, P, np.arange(5000))
    n = res["pages_needed"] + 7
    free = np.arange(n) if free_seed is None else np.random.default_rng(free_seed).permutation(n)
    res = oracle.reserve(ratio, ctxv, group_of, H // Hp, P, free)
    Nmax = int(ctxv.max())
    dk = rng.standard_normal((Bn, L, H, Nmax, d))
    dv = rng.standard_normal((Bn, L, H, Nmax, d))
    pool = np.full((n, 2, Hp, P, d), np.nan)      # unused slots poison any stray read
    write_dense(pool, dk, dv, res["kv_len"], res["offsets"], res["pages"], group_of, slot_of, L, H // Hp, P)
    q = rng.standard_normal((L, Bn, H * gqa, d))
    return dict(g=g, res=res, group_of=group_of, slot_of=slot_of, pool=pool, dk=dk, dv=dv, q=q, Bn=Bn, ctx=ctxv)


def _run_decode(c, layer, **kw):
    return oracle.decode_attention(c["q"][layer], c["pool"], layer, geom=c["g"], batch=c["Bn"],
                                   kv_len=c["res"]["kv_len"], offsets=c["res"]["offsets"], pages=c["res"]["pages"],
                                   group_of=c["group_of"], slot_of=c["slot_of"], **kw)


def test_decode_bruteforce_loops():
    c = small_case(1, Bn=2, L=2, H=2, gqa=2, d=4, Hp=1, P=4, ctx=(3, 8))
    for layer in range(2):
        O, lse = _run_decode(c, layer)
        scale = 1.0 / math.sqrt(4)
        for b in range(2):
            for qh in range(4):
                h = qh // 2
                n = c["res"]["kv_len"][b, layer, h]
                num = [0.0] * 4
                den = 0.0
                for t in range(n):
                    z = sum(c["q"][layer, b, qh, e] * c["dk"][b, layer, h, t, e] for e in range(4)) * scale
                    w = math.exp(z)                     # no max subtraction: tiny logits only
                    den += w
                    for e in range(4):
                        num[e] += w * c["dv"][b, layer, h, t, e]
                for e in range(4):
                    assert O[b, qh, e] == pytest.approx(num[e] / den, rel=1e-12, abs=1e-12)
                assert lse[b, qh] == pytest.approx(math.log(den), rel=1e-12, abs=1e-12)


def test_decode_full_ratio_equals_sdpa():
    Bn, L, H, gqa, d = 3, 1, 4, 3, 16
    c = small_case(2, Bn=Bn, L=L, H=H, gqa=gqa, d=d, Hp=2, P=4, ctx=(10, 50), ratio=np.ones((Bn, L, H)))
    O, _ = _run_decode(c, 0)
    for b in range(Bn):
        n = int(c["ctx"][b])
        q = torch.from_numpy(c["q"][0, b][:, None, :])                                  # [Hq][1][d]
        k = torch.from_numpy(c["dk"][b, 0, :, :n]).repeat_interleave(gqa, dim=0)       # [Hq][n][d]
        v = torch.from_numpy(c["dv"][b, 0, :, :n]).repeat_interleave(gqa, dim=0)
        ref = torch.nn.functional.scaled_dot_product_attention(q, k, v)[:, 0, :].numpy()
        np.testing.assert_allclose(O[b], ref, rtol=0, atol=1e-12)


def test_decode_single_retained_token_returns_its_value():
    Bn, L, H, gqa, d = 2, 1, 4, 2, 8
    c = small_case(3, Bn=Bn, L=L, H=H, gqa=gqa, d=d, Hp=2, P=4, ctx=(20, 30), ratio=np.full((Bn, L, H), 1e-6))
    assert np.all(c["res"]["kv_len"] == 1)
    O, lse = _run_decode(c, 0)
    for b in range(Bn):
        for qh in range(H * gqa):
            h = qh // gqa
            assert np.array_equal(O[b, qh], c["dv"][b, 0, h, 0])
            assert lse[b, qh] == pytest.approx(np.dot(c["q"][0, b, qh], c["dk"][b, 0, h, 0]) / math.sqrt(d), rel=1e-15)


def test_decode_placement_invariance_bitwise():
    a = small_case(4, free_seed=None)
    b = small_case(4, free_seed=99)
    assert not np.array_equal(a["res"]["pages"], b["res"]["pages"])
    for layer in range(2):
        Oa, la = _run_decode(a, layer)
        Ob, lb = _run_decode(b, layer)
        assert np.array_equal(Oa, Ob) and np.array_equal(la, lb)


@pytest.mark.parametrize("mode,n_bins,st", [(oracle.MODE_AOT, 5, 7), (oracle.MODE_AOT, 64, 300),
                                            (oracle.MODE_NAIVE, 1, 1), (oracle.MODE_UNIFORM, 40, 1),
                                            (oracle.MODE_FILL, 7, 1), (oracle.MODE_FILL, 100, 1)])
def test_decode_split_invariance(mode, n_bins, st):
    c = small_case(5, Bn=3, L=2, H=4, gqa=2, d=8, Hp=2, P=4, ctx=(30, 90))
    for layer in range(2):
        plan = oracle.partition_plan(c["res"]["kv_len"], c["res"]["offsets"], c["group_of"], c["slot_of"], layer,
                                     num_layers=2, num_groups=2, page_size=4, mode=mode, n_bins=n_bins,
                                     split_target=st)
        if mode == oracle.MODE_AOT and st >= 300:
            assert plan["num_partials"] > 0
        O, lse = _run_decode(c, layer)
        O2, lse2 = oracle.decode_by_plan(c["q"][layer], c["pool"], layer, plan, geom=c["g"], batch=c["Bn"],
                                         offsets=c["res"]["offsets"], pages=c["res"]["pages"],
                                         group_of=c["group_of"], slot_of=c["slot_of"])
        np.testing.assert_allclose(O2, O, rtol=0, atol=1e-12)
        np.testing.assert_allclose(lse2, lse, rtol=0, atol=1e-12)


# -------------------------------------------------------------- prefill

def test_prefill_chunk_of_one_equals_decode_over_one_more_key():
    """A one-token chunk is a decode step whose cache also holds that token."""
    Bn, L, H, gqa, d, Hp, P = 2, 1, 4, 2, 8, 2, 4
    c = small_case(6, Bn=Bn, L=L, H=H, gqa=gqa, d=d, Hp=Hp, P=P, ctx=(20, 40))
    hist = c["res"]["kv_len"]
    # decode-side cache: one more retained row per head, the chunk's own key
    longer = hist + 1
    G = H // Hp
    gl = np.zeros((Bn, L, G), dtype=np.int64)
    for b in range(Bn):
        for h in range(H):
            gl[b, 0, c["group_of"][0, h]] = max(gl[b, 0, c["group_of"][0, h]], longer[b, 0, h])
    npg = -(-gl // P)
    offsets = np.concatenate([[0], np.cumsum(npg.reshape(-1))])
    pages = np.arange(offsets[-1])
    pool2 = np.full((offsets[-1], 2, Hp, P, d), np.nan)
    write_dense(pool2, c["dk"], c["dv"], longer, offsets, pages, c["group_of"], c["slot_of"], L, G, P)
    q = c["q"][0][:, None]                                                  # [B][1][Hq][d]
    k_new = np.stack([c["dk"][b, 0, :, hist[b, 0, :]].diagonal().T for b in range(Bn)])[:, None]   # [B][1][H][d]
    v_new = np.stack([c["dv"][b, 0, :, hist[b, 0, :]].diagonal().T for b in range(Bn)])[:, None]
    for b in range(Bn):
        for h in range(H):
            assert np.array_equal(k_new[b, 0, h], c["dk"][b, 0, h, hist[b, 0, h]])
    Op = oracle.prefill_attention(q, k_new, v_new, c["pool"], 0, geom=c["g"], kv_len=hist,
                                  offsets=c["res"]["offsets"], pages=c["res"]["pages"],
                                  group_of=c["group_of"], slot_of=c["slot_of"])
    Od, _ = oracle.decode_attention(c["q"][0], pool2, 0, geom=c["g"], batch=Bn, kv_len=longer, offsets=offsets,
                                    pages=pages, group_of=c["group_of"], slot_of=c["slot_of"])
    np.testing.assert_allclose(Op[:, 0], Od, rtol=0, atol=1e-12)


def test_prefill_full_prefix_equals_masked_sdpa():
    """All ratios 1: the history is the whole prefix, so chunked prefill is
    ordinary causal attention of the chunk rows over prefix + chunk."""
    Bn, L, H, gqa, d, Hp, P, C = 2, 1, 2, 2, 8, 1, 4, 6
    c = small_case(7, Bn=Bn, L=L, H=H, gqa=gqa, d=d, Hp=Hp, P=P, ctx=(9, 17), ratio=np.ones((Bn, L, H)))
    rng = np.random.default_rng(70)
    q = rng.standard_normal((Bn, C, H * gqa, d))
    k_new = rng.standard_normal((Bn, C, H, d))
    v_new = rng.standard_normal((Bn, C, H, d))
    O = oracle.prefill_attention(q, k_new, v_new, c["pool"], 0, geom=c["g"], kv_len=c["res"]["kv_len"],
                                 offsets=c["res"]["offsets"], pages=c["res"]["pages"],
                                 group_of=c["group_of"], slot_of=c["slot_of"])
    for b in range(Bn):
        n = int(c["ctx"][b])
        for qh in range(H * gqa):
            h = qh // gqa
            keys = torch.from_numpy(np.concatenate([c["dk"][b, 0, h, :n], k_new[b, :, h]]))[None]
            vals = torch.from_numpy(np.concatenate([c["dv"][b, 0, h, :n], v_new[b, :, h]]))[None]
            mask = torch.zeros(C, n + C, dtype=torch.bool)
            for i in range(C):
                mask[i, : n + i + 1] = True          # explicit bottom-right causal mask
            ref = torch.nn.functional.scaled_dot_product_attention(torch.from_numpy(q[b, :, qh])[None], keys, vals,
                                                                   attn_mask=mask)[0].numpy()
            np.testing.assert_allclose(O[b, :, qh], ref, rtol=0, atol=1e-12)


# ------------------------------------------------------------- prefill schedule

def test_prefill_schedule_hand():
    """B=1, H=3, C=300, gqa=1, kv=[64, 200, 1], 2 XCDs, 256-row blocks, 64-key tiles.
    Row tiles 2: chunk tiles 4 (rows 0..255) and 5 (rows 256..299); history tiles 1, 4, 1.
    Unit costs 11, 17, 11 -> u1 on XCD0, u0 then u2 on XCD1 (loads 17, 22).
    XCD0 runs (1,1)=9 then (1,0)=8; XCD1 runs (0,1)=6, (2,1)=6, (0,0)=5, (2,0)=5."""
    kv = np.array([[[64, 200, 1]]])
    order, load = oracle.prefill_schedule(kv, 0, 300, 1, 2)
    assert order.tolist() == [3, 1, 2, 5, -1, 0, -1, 4]
    assert load == [17, 22]


@pytest.mark.parametrize("seed", range(6))
def test_prefill_schedule_invariants(seed):
    rng = np.random.default_rng(seed)
    B, H, gqa = int(rng.integers(1, 6)), int(rng.choice([1, 2, 4, 8])), int(rng.integers(1, 9))
    C = int(rng.integers(1, 700))
    n_xcd = int(rng.integers(1, 9))
    kv = rng.integers(0, 5000, size=(B, 2, H))
    order, load = oracle.prefill_schedule(kv, 1, C, gqa, n_xcd)
    row_tiles = -(-(C * gqa) // 256)
    codes = [c for c in order.tolist() if c >= 0]
    assert sorted(codes) == list(range(B * H * row_tiles))            # every block exactly once
    assert len(order) % n_xcd == 0
    xcd_of = {}
    for k, c in enumerate(order.tolist()):
        if c >= 0:
            xcd_of.setdefault(c // row_tiles, set()).add(k % n_xcd)
    assert all(len(v) == 1 for v in xcd_of.values())                 # a unit's row tiles share one XCD

    def cost(c):
        u, rt = divmod(c, row_tiles)
        b, h = divmod(u, H)
        i_last = min(C - 1, (min((rt + 1) * 256, C * gqa) - 1) // gqa)
        return -(-int(kv[b, 1, h]) // 64) + i_last // 64 + 1
    unit_cost = {}
    for c in codes:
        unit_cost[c // row_tiles] = unit_cost.get(c // row_tiles, 0) + cost(c)
    # Graham's LPT bound on the XCD loads
    assert sum(load) == sum(unit_cost.values())
    assert max(load) <= sum(load) / n_xcd + max(unit_cost.values())
    for x in range(n_xcd):                                            # longest first on every XCD
        seq = [cost(c) for c in order.tolist()[x::n_xcd] if c >= 0]
        assert seq == sorted(seq, reverse=True)
        assert all(c == -1 for c in order.tolist()[x::n_xcd][len(seq):])


def test_weighted_fill_plan_config1_hand():
    """Config 1 (units of 32, 16, 8, 4 pages per request, 120 pages), two bins
    weighted 1:2: cuts at 0, floor(120/3) = 40, 120.  Bin 0 = unit (0,0) whole
    and the first 8 pages of (0,1); bin 1 = the rest of (0,1) and every later
    unit.  (0,1) is the only split unit (partials 0 and 1)."""
    _, _, _, plan = _cfg1_plan(mode=oracle.MODE_FILL, n_bins=2, bin_weights=[1, 2])
    assert [list(it) for it in plan["items"]] == [
        [8, 0, 0, 1, 0, 512, -1], [8, 0, 1, 0, 0, 128, 0],
        [8, 0, 1, 0, 128, 256, 1], [0, 0, 2, 1, 0, 128, -1], [0, 0, 3, 0, 0, 64, -1],
        [48, 1, 0, 1, 0, 512, -1], [48, 1, 1, 0, 0, 256, -1], [40, 1, 2, 1, 0, 128, -1], [40, 1, 3, 0, 0, 64, -1]]
    assert plan["bin_offsets"].tolist() == [0, 2, 9]
    assert plan["num_partials"] == 2


@pytest.mark.parametrize("seed", range(5))
def test_weighted_fill_shares(seed):
    """Every bin holds floor/ceil of its weighted share of the pages, equal
    weights reproduce the unweighted plan, and the pieces tile every unit."""
    rng = np.random.default_rng(seed)
    c = _random_case(rng)
    res, L, G, P = c["res"], c["L"], c["G"], c["P"]
    n_bins = int(rng.integers(1, 60))
    w = rng.integers(1, 1000, size=n_bins)
    for layer in range(L):
        kw = dict(num_layers=L, num_groups=G, page_size=P, mode=oracle.MODE_FILL, n_bins=n_bins)
        plan = oracle.partition_plan(res["kv_len"], res["offsets"], c["group_of"], c["slot_of"], layer,
                                     bin_weights=w, **kw)
        pages = np.zeros(n_bins, dtype=np.int64)
        for k in range(n_bins):
            for it in plan["items"][plan["bin_offsets"][k]:plan["bin_offsets"][k + 1]]:
                pages[k] += -(-(it[5] - it[4]) // P)
        total = pages.sum()
        share = total * w / w.sum()
        assert np.all(np.abs(pages - share) < 1)
        assert total == sum(-(-int(x) // P) for x in res["kv_len"][:, layer, :].ravel())
        eq = oracle.partition_plan(res["kv_len"], res["offsets"], c["group_of"], c["slot_of"], layer,
                                   bin_weights=np.ones(n_bins, dtype=np.int64), **kw)
        base = oracle.partition_plan(res["kv_len"], res["offsets"], c["group_of"], c["slot_of"], layer, **kw)
        assert eq["items"] == base["items"] and eq["bin_offsets"].tolist() == base["bin_offsets"].tolist()


# ------------------------------------------- compression fused into prefill

COMP = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "compress_hand.json")))


def _scores(rows):
    return np.array([float(x) for x in rows], dtype=np.float32)


def _hand_cache(ratio):
    """Runs the two hand chunks through compress_chunk on a tiny paged cache whose entries store their
    context position, and returns (per-chunk kept, per-chunk count, cache positions of each head)."""
    g = Geometry(1, 2, 2, 2, 2, 2)
    cap = np.array(COMP["capacity"]).reshape(1, 1, 2)
    r = np.array(ratio, dtype=np.float64).reshape(1, 1, 2)
    budget = np.array([COMP["ratio"]], dtype=np.float64)
    perm, gof, sof = oracle.cluster_heads(budget, 2)
    gl = oracle.group_lengths(cap, gof, 1)
    npages = -(-int(gl[0, 0, 0]) // g.page_size)
    offsets, pages = np.array([0, npages]), np.arange(npages)
    pool = np.full((npages, 2, 2, g.page_size, g.head_dim), -1.0)
    C = COMP["chunk_len"]
    kept_all, counts = [], []
    for c in range(2):
        pos = np.arange(c * C, (c + 1) * C, dtype=np.float64)
        k_new = np.broadcast_to(pos[None, :, None, None], (1, C, 2, 2)).copy()
        scores = np.stack([_scores(s) for s in COMP["scores"][c]])[None]
        pool, kept, cur, cnt = oracle.compress_chunk(k_new, -k_new, scores, pool, 0, geom=g, ratio=r, capacity=cap,
                                                     chunk_start=[c * C], chunk_tokens=[C], offsets=offsets,
                                                     pages=pages, group_of=gof, slot_of=sof)
        kept_all.append(kept[0])
        counts.append(cnt[0].tolist())
    cache = []
    for h in range(2):
        n = sum(cnt[h] for cnt in counts)
        K, V = oracle.gather_head(pool, 0, 0, h, 0, n, geom=g, offsets=offsets, pages=pages, group_of=gof,
                                  slot_of=sof)
        assert np.array_equal(V, -K)
        cache.append(K[:, 0].astype(int).tolist())
    return kept_all, counts, cache


def test_compress_hand():
    kept, counts, cache = _hand_cache(COMP["ratio"])
    assert kept == COMP["kept"]
    assert counts == COMP["count"]
    assert cache == COMP["cache_positions"]
    for c in range(2):
        for h in range(2):
            cur, cnt = oracle.chunk_keep_range(COMP["ratio"][h], COMP["capacity"][h], c * 4, 4)
            assert [cur, cnt] == [COMP["cursor"][c][h], COMP["count"][c][h]]


def test_compress_hand_overflow_keeps_top_within_reservation():
    kept, counts, cache = _hand_cache(COMP["overflow_ratio"])
    assert counts == COMP["overflow_count"]
    assert kept == COMP["overflow_kept"]
    assert [len(x) for x in cache] == COMP["capacity"]


def _tiny_scores(rng, n):
    """Scores with many ties, signed zeros, infinities and NaNs."""
    s = rng.integers(-3, 4, size=n).astype(np.float32) / 2
    s[rng.random(n) < 0.1] = np.nan
    s[rng.random(n) < 0.1] = -0.0
    s[rng.random(n) < 0.05] = np.inf
    s[rng.random(n) < 0.05] = -np.inf
    return s


def _beats(s, t, u):
    """Does entry t rank above entry u (descending score, NaN lowest, lower index on ties)?"""
    a, b = float(s[t]), float(s[u])
    if math.isnan(a) or math.isnan(b):
        return (not math.isnan(a)) or (math.isnan(b) and t < u)
    return a > b or (a == b and t < u)


@pytest.mark.parametrize("seed", range(6))
def test_top_entries_brute_force(seed):
    rng = np.random.default_rng(seed)
    for _ in range(40):
        n = int(rng.integers(0, 12))
        s = _tiny_scores(rng, n)
        for k in range(n + 1):
            kept = oracle.top_entries(s, k)
            assert kept == sorted(set(kept)) and len(kept) == k
            drop = [u for u in range(n) if u not in kept]
            assert all(_beats(s, t, u) for t in kept for u in drop)


def test_top_entries_matches_library_selection():
    import heapq
    rng = np.random.default_rng(3)
    for _ in range(50):
        n = int(rng.integers(1, 300))
        s = (rng.integers(-20, 20, size=n) / 4).astype(np.float32)   # NaN-free, many ties
        k = int(rng.integers(0, n + 1))
        lib = sorted(heapq.nlargest(k, range(n), key=lambda t: (float(s[t]), -t)))
        assert oracle.top_entries(s, k) == lib
        assert oracle.top_entries(s, k) == sorted(np.argsort(-s, kind="stable")[:k].tolist())


def test_chunk_counts_fp64_pitfall():
    # 0.07*50 is 3.5000000000000004 and 0.07*100 is 7.000000000000001 in fp64
    assert oracle.chunk_keep_range(0.07, 8, 0, 100) == (0, 8)
    assert [oracle.chunk_keep_range(0.07, 8, c0, 50) for c0 in (0, 50)] == [(0, 4), (4, 4)]


@pytest.mark.parametrize("seed", range(4))
def test_chunk_counts_telescope_to_eq4(seed):
    """Whatever the chunking, the chunks of a context keep exactly ceil(r*N) entries in all, each
    chunk appends right after the previous one and keeps at most its own length."""
    rng = np.random.default_rng(seed)
    for _ in range(300):
        N = int(rng.integers(1, 5000))
        r = float(rng.choice([rng.uniform(0.001, 1.0), 1.0, 0.07, 0.29, 1 / 3]))
        cap = int(oracle.retained_lengths(np.array([[[r]]]), [N])[0, 0, 0])
        cuts = np.unique(np.concatenate([[0, N], rng.integers(0, N + 1, size=int(rng.integers(0, 6)))]))
        nxt = 0
        for c0, c1 in zip(cuts[:-1], cuts[1:]):
            cur, cnt = oracle.chunk_keep_range(r, cap, int(c0), int(c1 - c0))
            assert cur == nxt and 0 <= cnt <= c1 - c0
            nxt = cur + cnt
        assert nxt == cap == math.ceil(r * N)


@pytest.mark.parametrize("seed", range(4))
def test_overflow_caps_at_reservation_and_keeps_a_subset(seed):
    """A selection ratio above the reserved one fills the reservation exactly; a chunk that hits the
    cap keeps a subset of what it would keep uncapped (Top(k1) within Top(k2) for k1 <= k2)."""
    rng = np.random.default_rng(100 + seed)
    for _ in range(100):
        N = int(rng.integers(2, 400))
        r_res = float(rng.uniform(0.02, 0.9))
        r_sel = min(1.0, r_res + float(rng.uniform(0.01, 0.5)))
        cap = math.ceil(r_res * N)
        C = int(rng.integers(1, N + 1))
        total = 0
        for c0 in range(0, N, C):
            n = min(C, N - c0)
            s = _tiny_scores(rng, n)
            _, cnt = oracle.chunk_keep_range(r_sel, cap, c0, n)
            _, free_cnt = oracle.chunk_keep_range(r_sel, 10**9, c0, n)
            assert cnt <= free_cnt
            assert set(oracle.top_entries(s, cnt)) <= set(oracle.top_entries(s, free_cnt))
            total += cnt
        assert total == cap


def test_compress_one_chunk_is_eq4_and_lands_in_pages():
    """A single chunk holding the whole context keeps Top(ceil(r*N), s) (Eq. 4 itself), stored in
    ascending token order at the head's retained entries 0..count-1 (page layout of Section 4.2.1)."""
    rng = np.random.default_rng(11)
    g = Geometry(1, 4, 8, 8, 4, 2)
    B, C = 3, 37
    budget = rng.uniform(0.05, 1.0, size=(1, 4))
    ratio = np.broadcast_to(budget, (B, 1, 4)).copy()
    perm, gof, sof = oracle.cluster_heads(budget, 2)
    res = oracle.reserve(ratio, [C] * B, gof, 2, g.page_size, rng.permutation(200))
    pool = rng.standard_normal((200, 2, 2, g.page_size, g.head_dim))
    k_new = rng.standard_normal((B, C, 4, g.head_dim))
    v_new = rng.standard_normal((B, C, 4, g.head_dim))
    scores = _tiny_scores(rng, B * 4 * C).reshape(B, 4, C)
    out, kept, cur, cnt = oracle.compress_chunk(k_new, v_new, scores, pool, 0, geom=g, ratio=ratio,
                                                capacity=res["kv_len"], chunk_start=[0] * B, chunk_tokens=[C] * B,
                                                offsets=res["offsets"], pages=res["pages"], group_of=gof,
                                                slot_of=sof)
    for b in range(B):
        for h in range(4):
            n = math.ceil(float(budget[0, h]) * C)
            assert cur[b, h] == 0 and cnt[b, h] == n
            assert kept[b][h] == oracle.top_entries(scores[b, h], n)
            K, V = oracle.gather_head(out, b, 0, h, 0, n, geom=g, offsets=res["offsets"], pages=res["pages"],
                                      group_of=gof, slot_of=sof)
            assert np.array_equal(K, k_new[b, kept[b][h], h]) and np.array_equal(V, v_new[b, kept[b][h], h])
    # nothing outside the written entries changed
    touched = np.zeros(out.shape[:4], dtype=bool)
    for b in range(B):
        for h in range(4):
            for i in range(int(cnt[b, h])):
                p, s, r = oracle.token_location(b, 0, h, i, num_layers=1, num_groups=2, page_size=g.page_size,
                                                offsets=res["offsets"], pages=res["pages"], group_of=gof,
                                                slot_of=sof)
                touched[p, :, s, r] = True
    assert np.array_equal(out[~touched], pool[~touched])


def test_compress_plan_pieces_cover_every_kept_entry():
    rng = np.random.default_rng(5)
    B, L, H = 4, 2, 4
    ratio = rng.uniform(0.02, 1.0, size=(B, L, H))
    cap = oracle.retained_lengths(ratio, [900] * B)
    gof = np.array([[0, 0, 1, 1]] * L)
    sof = np.array([[0, 1, 0, 1]] * L)
    offsets = np.arange(B * L * 2 + 1) * 100
    starts, toks = [0, 300, 600, 850], [300, 300, 300, 50]
    for R in (1, 7, 64):
        items, cur, cnt = oracle.compress_plan(ratio, cap, starts, toks, offsets, gof, sof, 1, num_layers=L,
                                               num_groups=2, rows_per_item=R)
        seen = {}
        for base, b, h, slot, n, c0, c, r0, r1 in items:
            assert base == offsets[(b * L + 1) * 2 + gof[1, h]] and slot == sof[1, h] and n == toks[b]
            assert (c0, c) == (cur[b, h], cnt[b, h]) and 0 <= r0 < r1 <= c and r1 - r0 <= R
            seen.setdefault((b, h), []).append((r0, r1))
        assert [k for k in seen] == sorted(seen)
        for b in range(B):
            for h in range(H):
                spans = seen.get((b, h), [])
                assert sum(r1 - r0 for r0, r1 in spans) == cnt[b, h]
                assert all(s[1] == t[0] for s, t in zip(spans, spans[1:]))


# ------------------------------------------------ memory footprint of paging

FOOT = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "footprint_hand.json")))


def _footprint(budget, ctx, Hp, grouping, ratio=None, P=16):
    budget = np.asarray(budget, dtype=np.float64)
    L, H = budget.shape
    _, gof, _ = oracle.cluster_heads(budget, Hp, grouping)
    r = np.broadcast_to(budget, (len(ctx), L, H)) if ratio is None else ratio
    return oracle.memory_footprint(r, ctx, gof, H // Hp, Hp, P)


def test_footprint_hand():
    for key, slots in FOOT["ragged_slots"].items():
        hp, grouping = key.split("-")
        f = _footprint(FOOT["budget"], FOOT["ctx_len"], int(hp),
                       oracle.GROUP_CLUSTERED if grouping == "clustered" else oracle.GROUP_ADJACENT)
        assert f["ragged_slots"] == slots and f["ragged_pages"] == FOOT["ragged_pages"][key], key
        assert f["full_slots"] == FOOT["full_slots"] and f["retained_slots"] == FOOT["retained_slots"]
        assert f["monolithic_slots"] == FOOT["monolithic_slots"]


def test_footprint_hand_partial_pages():
    c = FOOT["case2"]
    for key, slots in c["ragged_slots"].items():
        hp, grouping = key.split("-")
        f = _footprint(FOOT["budget"], c["ctx_len"], int(hp),
                       oracle.GROUP_CLUSTERED if grouping == "clustered" else oracle.GROUP_ADJACENT)
        assert f["ragged_slots"] == slots, key
        assert (f["full_slots"], f["retained_slots"], f["monolithic_slots"]) == \
            (c["full_slots"], c["retained_slots"], c["monolithic_slots"])


def test_footprint_config1_hand():
    # config 1: lengths {512, 256, 128, 64}; groups {3,2} (GL 128, 8 pages) and {1,0} (GL 512, 32 pages)
    f = _footprint(GOLD["budget"], GOLD["ctx_len"], 2, oracle.GROUP_CLUSTERED, P=16)
    assert f["ragged_pages"] == 80 and f["ragged_slots"] == 80 * 16 * 2
    assert f["full_slots"] == f["monolithic_slots"] == 2 * 32 * 16 * 4     # head 0 keeps everything
    assert f["retained_slots"] == 2 * (512 + 256 + 128 + 64)


@pytest.mark.parametrize("seed", range(5))
def test_clustering_minimises_ragged_slots_bruteforce(seed):
    """Without per-request jitter, retained lengths follow the budget order, so the clustered groups take
    the smallest possible group maxima: no equal-size partition of the heads allocates fewer slots."""
    rng = np.random.default_rng(seed)
    for _ in range(6):
        H = int(rng.choice([4, 6, 8]))
        Hp = int(rng.choice([h for h in (2, 3, 4) if H % h == 0]))
        budget = rng.choice([0.02, 0.1, 0.3, 0.6, 1.0], size=(1, H))
        ctx = rng.integers(1, 3000, size=3)
        P = int(rng.choice([1, 16]))
        best = _footprint(budget, ctx, Hp, oracle.GROUP_CLUSTERED, P=P)["ragged_slots"]
        ratio = np.broadcast_to(budget, (3, 1, H))
        kv = oracle.retained_lengths(ratio, ctx)

        def partitions(items):
            if not items:
                yield []
                return
            first, rest = items[0], items[1:]
            for others in itertools.combinations(rest, Hp - 1):
                left = [x for x in rest if x not in others]
                for tail in partitions(left):
                    yield [(first,) + others] + tail

        for part in partitions(list(range(H))):
            slots = 0
            for b in range(3):
                for grp in part:
                    slots += -(-max(int(kv[b, 0, h]) for h in grp) // P) * P * Hp
            assert best <= slots


@pytest.mark.parametrize("seed", range(3))
def test_footprint_orderings(seed):
    """retained <= ragged(H_p = 1) <= ragged(any H_p, any grouping) <= monolithic <= full."""
    rng = np.random.default_rng(40 + seed)
    L, H, B = 3, 8, 4
    budget = rng.uniform(0.02, 1.0, size=(L, H))
    ratio = np.clip(budget[None] + rng.uniform(-0.03, 0.03, size=(B, L, H)), 0.02, 1.0)
    ctx = rng.integers(100, 5000, size=B)
    one = _footprint(budget, ctx, 1, oracle.GROUP_CLUSTERED, ratio=ratio)
    for Hp in (1, 2, 4, 8):
        for grouping in (oracle.GROUP_CLUSTERED, oracle.GROUP_ADJACENT):
            f = _footprint(budget, ctx, Hp, grouping, ratio=ratio)
            assert f["retained_slots"] <= one["ragged_slots"] <= f["ragged_slots"] <= f["monolithic_slots"] \
                <= f["full_slots"]
            assert f["page_tables"] == B * L * H // Hp
            res = oracle.reserve(ratio, ctx, oracle.cluster_heads(budget, Hp, grouping)[1], H // Hp, 16,
                                 np.arange(10**6))
            assert res["pages_needed"] == f["ragged_pages"]


# ----------------------------------------- decode steps: append and plan reuse

def test_reserve_headroom_config1_hand():
    """Config 1 with room for 20 decode tokens: group {3,2} (GL 128) takes ceil(148/16) = 10 pages and group
    {1,0} (GL 512) ceil(532/16) = 34, so the tables start at 0, 10, 44, 54 and hold 88 pages."""
    budget, ratio, ctx = cfg1_arrays()
    _, gof, _ = oracle.cluster_heads(budget, 2)
    res = oracle.reserve(ratio, ctx, gof, 2, 16, np.arange(100), headroom=[20, 20])
    assert res["offsets"].tolist() == [0, 10, 44, 54, 88]
    assert res["kv_len"].tolist() == GOLD["kv_len"]


def _tiny_decode_case(seed, T, mode, Hp=2):
    rng = np.random.default_rng(seed)
    g = Geometry(2, 4, 8, 8, 4, Hp)
    B = 3
    budget = rng.uniform(0.05, 1.0, size=(2, 4))
    ratio = np.clip(budget[None] + rng.uniform(-0.03, 0.03, size=(B, 2, 4)), 0.02, 1.0)
    ctx = rng.integers(5, 60, size=B)
    _, gof, sof = oracle.cluster_heads(budget, Hp)
    res = oracle.reserve(ratio, ctx, gof, g.num_groups, g.page_size, rng.permutation(400), headroom=[T] * B)
    pool = rng.standard_normal((400, 2, Hp, g.page_size, g.head_dim))
    return rng, g, B, gof, sof, res, pool


@pytest.mark.parametrize("mode", [oracle.MODE_AOT, oracle.MODE_NAIVE, oracle.MODE_UNIFORM, oracle.MODE_FILL])
def test_open_plan_marks_exactly_the_last_chunk_of_each_unit(mode):
    _, g, B, gof, sof, res, _ = _tiny_decode_case(3, 9, mode)
    kw = dict(num_layers=2, num_groups=g.num_groups, page_size=g.page_size, mode=mode, n_bins=5, split_target=11)
    closed = oracle.partition_plan(res["kv_len"], res["offsets"], gof, sof, 1, **kw)
    opened = oracle.partition_plan(res["kv_len"], res["offsets"], gof, sof, 1, open_end=True, **kw)
    assert len(closed["items"]) == len(opened["items"])
    ends = {}
    for c, o in zip(closed["items"], opened["items"]):
        assert c[:5] == o[:5] and c[6] == o[6]
        if o[5] < 0:
            b, h = o[1], o[2]
            t = (b * 2 + 1) * g.num_groups + gof[1, h]
            assert c[5] == res["kv_len"][b, 1, h] and -o[5] == (res["offsets"][t + 1] - res["offsets"][t]) * 4
            assert (b, h) not in ends
            ends[(b, h)] = o
        else:
            assert o[5] == c[5] < res["kv_len"][o[1], 1, o[2]]
    assert len(ends) == B * 4


@pytest.mark.parametrize("mode", [oracle.MODE_AOT, oracle.MODE_NAIVE, oracle.MODE_UNIFORM, oracle.MODE_FILL])
def test_plan_from_step_zero_serves_later_steps(mode):
    """A plan built before the first decode step, with open ends, gives the plain attention over the grown
    cache after T appended tokens (split-KV merge exact in fp64); the appended rows read back in order."""
    T = 9
    rng, g, B, gof, sof, res, pool = _tiny_decode_case(7, T, mode)
    kw = dict(num_layers=2, num_groups=g.num_groups, page_size=g.page_size, mode=mode, n_bins=5, split_target=11)
    plan = oracle.partition_plan(res["kv_len"], res["offsets"], gof, sof, 1, open_end=True, **kw)
    live = res["kv_len"].copy()
    toks = []
    for _ in range(T):
        kt, vt = rng.standard_normal((B, 4, g.head_dim)), rng.standard_normal((B, 4, g.head_dim))
        pool, live, full = oracle.append_token(kt, vt, pool, 1, geom=g, live_len=live, offsets=res["offsets"],
                                               pages=res["pages"], group_of=gof, slot_of=sof)
        assert full == []
        toks.append((kt, vt))
    assert np.array_equal(live[:, 1], res["kv_len"][:, 1] + T) and np.array_equal(live[:, 0], res["kv_len"][:, 0])
    for b in range(B):
        for h in range(4):
            n = int(res["kv_len"][b, 1, h])
            K, V = oracle.gather_head(pool, b, 1, h, n, n + T, geom=g, offsets=res["offsets"], pages=res["pages"],
                                      group_of=gof, slot_of=sof)
            assert np.array_equal(K, np.stack([t[0][b, h] for t in toks]))
            assert np.array_equal(V, np.stack([t[1][b, h] for t in toks]))
    q = rng.standard_normal((B, 8, g.head_dim))
    ref, ref_lse = oracle.decode_attention(q, pool, 1, geom=g, batch=B, kv_len=live, offsets=res["offsets"],
                                           pages=res["pages"], group_of=gof, slot_of=sof)
    got, got_lse = oracle.decode_by_plan(q, pool, 1, plan, geom=g, batch=B, offsets=res["offsets"],
                                         pages=res["pages"], group_of=gof, slot_of=sof, live_len=live)
    assert np.abs(got - ref).max() < 1e-12 and np.abs(got_lse - ref_lse).max() < 1e-12


def test_append_without_room_writes_nothing():
    """Config 1 reserved without headroom: heads 0 (512 of 512) and 2 (128 of 128) have no room for a decode
    token, heads 1 and 3 do."""
    budget, ratio, ctx = cfg1_arrays()
    g = Geometry(1, 4, 8, 64, 16, 2)
    _, gof, sof = oracle.cluster_heads(budget, 2)
    res = oracle.reserve(ratio, ctx, gof, 2, 16, np.arange(100))
    pool = np.zeros((100, 2, 2, 16, 64))
    k = np.ones((2, 4, 64))
    out, live, full = oracle.append_token(k, -k, pool, 0, geom=g, live_len=res["kv_len"], offsets=res["offsets"],
                                          pages=res["pages"], group_of=gof, slot_of=sof)
    assert full == [(0, 0), (0, 2), (1, 0), (1, 2)]
    assert (live - res["kv_len"]).tolist() == [[[0, 1, 0, 1]], [[0, 1, 0, 1]]]
    assert int((out != 0).sum()) == 2 * 2 * 2 * 64      # two heads of two requests, a K and a V row each


# ------------------------------------------ Algorithm 1's split map executed as is

def test_split_map_plan_config1_hand():
    """Config 1 at N_CTA = 8: S = [2, 6].  Group {3,2}: units b0h2 (8 pages), b0h3 (4), b1h2 (8), b1h3 (4),
    24 pages in 2 bins of 12.  Group {1,0}: b0h0 (32), b0h1 (16), b1h0 (32), b1h1 (16), 96 pages in 6 bins of
    16, so each 512-token head is split in two (partials 0-1 and 2-3)."""
    budget, ratio, ctx = cfg1_arrays()
    perm, gof, sof = oracle.cluster_heads(budget, 2)
    res = oracle.reserve(ratio, ctx, gof, 2, 16, np.arange(100))
    S = oracle.split_map(budget, perm, 2, 8)
    assert S.tolist() == [[2, 6]]
    pl = oracle.partition_plan(res["kv_len"], res["offsets"], gof, sof, 0, num_layers=1, num_groups=2, page_size=16,
                               mode=oracle.MODE_SPLIT_MAP, bin_weights=S[0])
    # (pt_base, b, h, slot, t0, t1, out_idx); group 0 tables start at 0 and 40, group 1 at 8 and 48
    assert pl["items"] == [(0, 0, 2, 1, 0, 128, -1), (0, 0, 3, 0, 0, 64, -1),
                           (40, 1, 2, 1, 0, 128, -1), (40, 1, 3, 0, 0, 64, -1),
                           (8, 0, 0, 1, 0, 256, 0), (8, 0, 0, 1, 256, 512, 1), (8, 0, 1, 0, 0, 256, -1),
                           (48, 1, 0, 1, 0, 256, 2), (48, 1, 0, 1, 256, 512, 3), (48, 1, 1, 0, 0, 256, -1)]
    assert pl["bin_offsets"].tolist() == [0, 2, 4, 5, 6, 7, 8, 9, 10]
    assert pl["bin_load"].tolist() == [192, 192] + [256] * 6


@pytest.mark.parametrize("seed", range(4))
def test_split_map_plan_with_one_group_is_the_fill_plan(seed):
    """With H_p = H there is one group per layer, whose S bins cut the whole layer: the sequential-fill plan
    with S bins (two separately written constructions)."""
    rng = np.random.default_rng(seed)
    L, H, B = 2, 4, 3
    budget = rng.uniform(0.05, 1.0, size=(L, H))
    ratio = np.clip(budget[None] + rng.uniform(-0.03, 0.03, size=(B, L, H)), 0.02, 1.0)
    perm, gof, sof = oracle.cluster_heads(budget, H)
    res = oracle.reserve(ratio, rng.integers(10, 900, size=B), gof, 1, 8, np.arange(10**4))
    for n_cta in (1, 5, 37):
        S = oracle.split_map(budget, perm, H, n_cta)
        for l in range(L):
            kw = dict(num_layers=L, num_groups=1, page_size=8)
            a = oracle.partition_plan(res["kv_len"], res["offsets"], gof, sof, l, mode=oracle.MODE_SPLIT_MAP,
                                      bin_weights=S[l], **kw)
            b = oracle.partition_plan(res["kv_len"], res["offsets"], gof, sof, l, mode=oracle.MODE_FILL,
                                      n_bins=int(S[l, 0]), **kw)
            assert a["items"] == b["items"] and a["bin_offsets"].tolist() == b["bin_offsets"].tolist()


def test_split_map_plan_decodes_exactly():
    rng = np.random.default_rng(12)
    g = Geometry(1, 4, 8, 8, 4, 2)
    B = 3
    budget = rng.uniform(0.05, 1.0, size=(1, 4))
    ratio = np.clip(budget[None] + rng.uniform(-0.03, 0.03, size=(B, 1, 4)), 0.02, 1.0)
    perm, gof, sof = oracle.cluster_heads(budget, 2)
    res = oracle.reserve(ratio, rng.integers(5, 90, size=B), gof, 2, 4, rng.permutation(300))
    pool = rng.standard_normal((300, 2, 2, 4, 8))
    q = rng.standard_normal((B, 8, 8))
    S = oracle.split_map(budget, perm, 2, 11)
    pl = oracle.partition_plan(res["kv_len"], res["offsets"], gof, sof, 0, num_layers=1, num_groups=2, page_size=4,
                               mode=oracle.MODE_SPLIT_MAP, bin_weights=S[0])
    ref, _ = oracle.decode_attention(q, pool, 0, geom=g, batch=B, kv_len=res["kv_len"], offsets=res["offsets"],
                                     pages=res["pages"], group_of=gof, slot_of=sof)
    got, _ = oracle.decode_by_plan(q, pool, 0, pl, geom=g, batch=B, offsets=res["offsets"], pages=res["pages"],
                                   group_of=gof, slot_of=sof)
    assert np.abs(got - ref).max() < 1e-12
    assert len(pl["bin_offsets"]) - 1 == int(S.sum())


# ------------------------------------------------ calibration and request lifecycle

def test_implicit_ratios_hand():
    """L = 1, H = 2, N = 4, rho = 0.5: the layer keeps ceil(0.5*8) = 4 of the flattened scores.  0.9 (h0 t0) and
    0.8 (h1 t1) come first; three entries tie at 0.5 (h0 t2, h0 t3, h1 t0) and the two lower flattened indices
    (both in head 0) win, so head 0 keeps 3 of 4 and head 1 keeps 1 of 4."""
    sc = np.array([[[0.9, 0.1, 0.5, 0.5], [0.5, 0.8, 0.0, -0.0]]], dtype=np.float32)
    r, c = oracle.implicit_ratios(sc, 0.5)
    assert c.tolist() == [[3, 1]] and r.tolist() == [[0.75, 0.25]]


def test_implicit_ratios_reduce_to_uniform_when_heads_agree():
    """Identical heads with distinct scores: the global selection keeps rho*N entries of every head when rho*H*N
    is a multiple of H (the uniform compression of Eq. 2)."""
    rng = np.random.default_rng(2)
    N, H = 40, 4
    row = rng.permutation(N).astype(np.float32)
    sc = np.broadcast_to(row, (1, H, N)).copy()
    for rho in (0.25, 0.5, 0.75, 1.0):
        r, c = oracle.implicit_ratios(sc, rho)
        assert c.tolist() == [[int(rho * N)] * H]
        kept = oracle.top_entries(row, int(rho * N))
        assert set(kept) == set(np.argsort(-row)[: int(rho * N)].tolist())


@pytest.mark.parametrize("seed", range(4))
def test_implicit_ratios_brute_force(seed):
    rng = np.random.default_rng(seed)
    for _ in range(20):
        L, H, N = 1, int(rng.integers(1, 4)), int(rng.integers(1, 7))
        sc = _tiny_scores(rng, L * H * N).reshape(L, H, N)
        rho = float(rng.choice([0.1, 0.3, 0.5, 1.0, rng.uniform(0.01, 1.0)]))
        r, c = oracle.implicit_ratios(sc, rho)
        k = math.ceil(rho * H * N)
        assert int(c.sum()) == k
        flat = sc.reshape(-1)
        # some kept set of these per-head counts must beat every dropped entry: check via the sorted order
        order = sorted(range(H * N), key=lambda i: (1, 0.0, i) if math.isnan(float(flat[i])) else (0, -float(flat[i]), i))
        kept = set(order[:k])
        assert all(_beats(flat, t, u) for t in kept for u in range(H * N) if u not in kept)
        assert [sum(1 for i in kept if i // N == h) for h in range(H)] == c[0].tolist()


def test_calibrated_budget_hand_and_cases():
    # two samples 0.2 and 0.4: mu = 0.3, population sigma = 0.1, alpha = 2 -> 0.5 (the sample standard deviation
    # would give 0.583)
    B = oracle.calibrate_budget(np.array([[[0.2]], [[0.4]]]), 2.0, 0.01)
    assert abs(B[0, 0] - 0.5) < 1e-15
    samples = np.array([[[0.1, 0.9, 0.0]], [[0.3, 0.95, 0.0]], [[0.2, 0.85, 0.0]]])
    B0 = oracle.calibrate_budget(samples, 0.0, 0.01)
    assert np.allclose(B0, [[0.2, 0.9, 0.01]], rtol=0, atol=1e-15)          # alpha 0: the mean; a never-kept head: floor
    assert oracle.calibrate_budget(samples, 3.0, 0.01)[0, 1] == 1.0          # 0.9 + 3 * 0.0408 > 1: capped
    one = oracle.calibrate_budget(samples[:1], 3.0, 0.01)
    assert one.tolist() == [[0.1, 0.9, 0.01]]                                # one sample: sigma = 0


def test_calibrated_budgets_sum_to_the_global_budget():
    """With alpha = 0 and one sample, the per-head budgets keep the layer's global count up to rounding:
    sum_h ceil(B_h * N) lies within [ceil(rho*H*N), ceil(rho*H*N) + H]."""
    rng = np.random.default_rng(8)
    for _ in range(10):
        L, H, N = 2, 4, int(rng.integers(20, 200))
        sc = rng.standard_normal((L, H, N)).astype(np.float32) * rng.uniform(0.2, 3.0, size=(1, H, 1))
        rho = float(rng.uniform(0.1, 0.9))
        r, _ = oracle.implicit_ratios(sc, rho)
        B = oracle.calibrate_budget(r[None], 0.0, 1e-9)
        k = math.ceil(rho * H * N)
        for l in range(L):
            tot = sum(math.ceil(float(B[l, h]) * N) for h in range(H))
            assert k <= tot <= k + H


def test_release_and_readmit_config1_hand():
    budget, ratio, ctx = cfg1_arrays()
    _, gof, _ = oracle.cluster_heads(budget, 2)
    res = oracle.reserve(ratio, ctx, gof, 2, 16, np.arange(100))
    assert res["offsets"].tolist() == [0, 8, 40, 48, 80]
    freed, off, pages = oracle.release_requests(res["offsets"], res["pages"], [True, False], 1, 2)
    assert freed.tolist() == list(range(40)) and off.tolist() == [0, 8, 40] and pages.tolist() == list(range(40, 80))
    freed, off, pages = oracle.release_requests(res["offsets"], res["pages"], [False, True], 1, 2)
    assert freed.tolist() == list(range(40, 80)) and off.tolist() == [0, 8, 40] and pages.tolist() == list(range(40))
    # readmit the released request from the freed pages: the batch's tables hold every page once again
    again = oracle.reserve(ratio[1:], ctx[1:], gof, 2, 16, freed)
    o2, p2 = oracle.concat_tables(off, pages, again["offsets"], again["pages"])
    assert o2.tolist() == res["offsets"].tolist() and sorted(p2.tolist()) == list(range(80))


@pytest.mark.parametrize("seed", range(3))
def test_release_invariants(seed):
    rng = np.random.default_rng(seed)
    L, H, B = 2, 4, 6
    budget = rng.uniform(0.05, 1.0, size=(L, H))
    _, gof, _ = oracle.cluster_heads(budget, 2)
    ratio = np.broadcast_to(budget, (B, L, H))
    ctx = rng.integers(1, 500, size=B)
    res = oracle.reserve(ratio, ctx, gof, 2, 16, rng.permutation(10**4))
    fin = rng.random(B) < 0.5
    freed, off, pages = oracle.release_requests(res["offsets"], res["pages"], fin, L, 2)
    assert sorted(freed.tolist() + pages.tolist()) == sorted(res["pages"].tolist())
    survivors = [b for b in range(B) if not fin[b]]
    sizes = np.diff(res["offsets"]).reshape(B, L * 2)
    assert np.diff(off).tolist() == sizes[survivors].reshape(-1).tolist()
