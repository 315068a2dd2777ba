"""libtangram.so host integer calls vs the fp64 oracle, bit for bit (CPU only).

Covers Budget-Aware Clustering (Section 4.2.2), Budget Reservation and the
ragged per-group page tables (Eq. 4, Sections 4.1 and 4.2.1), Algorithm 1's
split map and the balanced partition plan, plus the error contract of
include/tangram.h.
"""
import json
import os

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import oracle
from paper_2606_06302_amd import tangram as tg
from workloads import Geometry, config, free_list, pool_pages_for

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "config1_hand.json")))


def _items_as_tuples(items):
    return [tuple(int(x) for x in it) for it in items.tolist()]


def _full_compare(geom, batch, ctx, ratio, budget, free, pool, grouping=0, mode=0, n_bins=7, split_target=33,
                  layers=None, bin_weights=None):
    L, H, Hp = geom.num_layers, geom.num_kv_heads, geom.heads_per_group
    G = H // Hp
    perm, gof, sof = tg.tg_cluster_heads(geom, budget, grouping)
    operm, ogof, osof = oracle.cluster_heads(budget, Hp, grouping)
    assert np.array_equal(perm, operm) and np.array_equal(gof, ogof) and np.array_equal(sof, osof)
    res = tg.tg_reserve(geom, ctx, ratio, budget, gof, free, pool)
    ores = oracle.reserve(ratio if ratio is not None else np.broadcast_to(budget, (batch, L, H)), ctx, ogof, G,
                          geom.page_size, free)
    assert np.array_equal(res["kv_len"], ores["kv_len"])
    assert np.array_equal(res["group_len"], ores["group_len"])
    assert np.array_equal(res["pt_offsets"], ores["offsets"])
    assert np.array_equal(res["pt_pages"], ores["pages"])
    assert res["pages_needed"] == ores["pages_needed"]
    for n_cta in (1, 8, 256, 1024):
        assert np.array_equal(tg.tg_split_map(geom, budget, perm, n_cta), oracle.split_map(budget, operm, Hp, n_cta))
    for layer in (range(L) if layers is None else layers):
        pl = tg.tg_build_plan(geom, batch, layer, res["kv_len"], res["pt_offsets"], gof, sof, mode, n_bins,
                              split_target, bin_weights=bin_weights)
        opl = oracle.partition_plan(ores["kv_len"], ores["offsets"], ogof, osof, layer, num_layers=L, num_groups=G,
                                    page_size=geom.page_size, mode=mode, n_bins=n_bins, split_target=split_target,
                                    bin_weights=bin_weights)
        assert _items_as_tuples(pl["items"]) == opl["items"]
        assert pl["bin_offsets"].tolist() == opl["bin_offsets"].tolist()
        assert np.array_equal(pl["unit_splits"], opl["unit_splits"])
        assert np.array_equal(pl["unit_partial_base"], opl["unit_partial_base"])
        assert pl["num_partials"] == opl["num_partials"]
    return res


def test_config1_matches_hand_values_and_oracle():
    wl = config(1)
    res = _full_compare(wl.geom, wl.batch, wl.ctx_len, wl.ratio, wl.budget, np.arange(100, dtype=np.int32), 100,
                        n_bins=8, split_target=16)
    assert res["pt_offsets"].tolist() == GOLD["offsets"]
    gof = tg.tg_cluster_heads(wl.geom, wl.budget)[1]
    pl = tg.tg_build_plan(wl.geom, 2, 0, res["kv_len"], res["pt_offsets"], gof,
                          tg.tg_cluster_heads(wl.geom, wl.budget)[2], 0, 8, 16)
    assert [list(t) for t in _items_as_tuples(pl["items"])] == GOLD["plan_split_target16_bins8"]["items"]
    fill = tg.tg_build_plan(wl.geom, 2, 0, res["kv_len"], res["pt_offsets"], gof,
                            tg.tg_cluster_heads(wl.geom, wl.budget)[2], tg.TG_PLAN_AOT_FILL, 8, 1)
    assert [list(t) for t in _items_as_tuples(fill["items"])] == GOLD["plan_fill_bins8"]["items"]
    assert fill["bin_offsets"].tolist() == GOLD["plan_fill_bins8"]["bin_offsets"]


@pytest.mark.parametrize("cfg", [1, 2, 4, 5])
def test_workload_configs_bit_exact(cfg):
    wl = config(cfg)
    gof = tg.tg_cluster_heads(wl.geom, wl.budget)[1]
    need = tg.tg_reserve(wl.geom, wl.ctx_len, wl.ratio, None, gof, np.zeros(0, np.int32), 0, size_query=True)
    pool = pool_pages_for(need["pages_needed"])
    free = free_list(wl, pool)
    for mode, nb, stg in [(0, 512, 2048), (1, 1, 1), (2, 512, 1), (3, 512, 1)]:
        _full_compare(wl.geom, wl.batch, wl.ctx_len, wl.ratio, wl.budget, free, pool, mode=mode, n_bins=nb,
                      split_target=stg)


@pytest.mark.slow
def test_config3_tables_and_two_layers_bit_exact():
    wl = config(3)
    gof = tg.tg_cluster_heads(wl.geom, wl.budget)[1]
    need = tg.tg_reserve(wl.geom, wl.ctx_len, wl.ratio, None, gof, np.zeros(0, np.int32), 0, size_query=True)
    pool = pool_pages_for(need["pages_needed"])
    _full_compare(wl.geom, wl.batch, wl.ctx_len, wl.ratio, wl.budget, free_list(wl, pool), pool, n_bins=512,
                  split_target=2048, layers=[0, 37])


@settings(max_examples=60, deadline=None)
@given(st.data())
def test_random_geometries_bit_exact(data):
    H = data.draw(st.sampled_from([1, 2, 3, 4, 6, 8, 12, 16]))
    Hp = data.draw(st.sampled_from([d for d in range(1, H + 1) if H % d == 0]))
    L = data.draw(st.integers(1, 3))
    B = data.draw(st.integers(1, 4))
    P = data.draw(st.sampled_from([1, 4, 16]))
    geom = Geometry(L, H, H * data.draw(st.integers(1, 3)), 8, P, Hp)
    grid = data.draw(st.booleans())
    shape = (L, H)
    rng = np.random.default_rng(data.draw(st.integers(0, 2**31)))
    if grid:   # ties and exact binary fractions
        budget = rng.integers(1, 9, size=shape) / 8.0
    else:
        budget = rng.uniform(1e-3, 1.0, size=shape)
    use_ratio = data.draw(st.booleans())
    ratio = np.clip(budget[None] + rng.uniform(-.03, .03, size=(B, L, H)), 0.02, 1.0) if use_ratio else None
    ctx = rng.integers(1, 500, size=B).astype(np.int32)
    grouping = data.draw(st.sampled_from([0, 1]))
    gof = tg.tg_cluster_heads(geom, budget, grouping)[1]
    need = tg.tg_reserve(geom, ctx, ratio, budget, gof, np.zeros(0, np.int32), 0, size_query=True)["pages_needed"]
    pool = need + int(rng.integers(0, 30))
    free = rng.permutation(pool).astype(np.int32)
    mode = data.draw(st.sampled_from([0, 1, 2, 3]))
    n_bins = data.draw(st.integers(1, 64))
    weights = None
    if mode == 3 and data.draw(st.booleans()):
        weights = rng.integers(1, data.draw(st.sampled_from([2, 1000, 65536])), size=n_bins).astype(np.int32)
    _full_compare(geom, B, ctx, ratio, budget, free, pool, grouping=grouping, mode=mode,
                  n_bins=n_bins, split_target=data.draw(st.integers(1, 300)), bin_weights=weights)


def test_fp64_ceil_pitfalls_match_oracle():
    geom = Geometry(1, 2, 2, 8, 16, 1)
    budget = np.array([[0.07, 0.29]])
    gof = tg.tg_cluster_heads(geom, budget)[1]
    res = tg.tg_reserve(geom, [100], None, budget, gof, np.arange(10, dtype=np.int32), 10)
    assert res["kv_len"].tolist() == [[[8, 29]]]


# ----------------------------------------------------------------- errors

def _geom1():
    return Geometry(1, 4, 8, 64, 16, 2)


@pytest.mark.parametrize("bad", [0.0, -1.0, 1.5, float("nan")])
def test_bad_budget_rejected(bad):
    b = np.array([[0.5, bad, 0.2, 0.1]])
    with pytest.raises(tg.TangramError) as e:
        tg.tg_cluster_heads(_geom1(), b)
    assert e.value.code == tg.TG_ERR_INVALID_ARG


def test_indivisible_groups_rejected():
    with pytest.raises(tg.TangramError) as e:
        tg.tg_cluster_heads(Geometry(1, 6, 6, 64, 16, 4), np.full((1, 6), .5))
    assert e.value.code == tg.TG_ERR_INVALID_ARG
    assert "heads_per_group" in tg.tg_last_error()


def test_out_of_pages_consumes_nothing():
    wl = config(1)
    gof = tg.tg_cluster_heads(wl.geom, wl.budget)[1]
    free = np.arange(79, dtype=np.int32)
    before = free.copy()
    with pytest.raises(tg.TangramError) as e:
        tg.tg_reserve(wl.geom, wl.ctx_len, wl.ratio, None, gof, free, 100)
    assert e.value.code == tg.TG_ERR_OUT_OF_PAGES and np.array_equal(free, before)


@pytest.mark.parametrize("free", [[0, 1, 1] + list(range(2, 90)), [-1] + list(range(1, 90)), list(range(80)) + [200]])
def test_bad_page_ids_rejected(free):
    wl = config(1)
    gof = tg.tg_cluster_heads(wl.geom, wl.budget)[1]
    free = np.array(free, dtype=np.int32)
    if free[-1] == 200:        # an out-of-pool id that is consumed
        free = np.concatenate([[200], np.arange(79)]).astype(np.int32)
    with pytest.raises(tg.TangramError) as e:
        tg.tg_reserve(wl.geom, wl.ctx_len, wl.ratio, None, gof, free, 100)
    assert e.value.code == tg.TG_ERR_INVALID_ARG


def test_plan_rejects_length_beyond_table():
    wl = config(1)
    perm, gof, sof = tg.tg_cluster_heads(wl.geom, wl.budget)
    res = tg.tg_reserve(wl.geom, wl.ctx_len, wl.ratio, None, gof, np.arange(100, dtype=np.int32), 100)
    kv = res["kv_len"].copy()
    kv[0, 0, 2] = 129        # head 2's group holds 8 pages = 128 rows
    with pytest.raises(tg.TangramError) as e:
        tg.tg_build_plan(wl.geom, 2, 0, kv, res["pt_offsets"], gof, sof, 0, 8, 16)
    assert e.value.code == tg.TG_ERR_INVALID_ARG


def test_status_strings_and_version():
    assert tg.tg_status_string(0) == "ok"
    assert tg.tg_status_string(tg.TG_ERR_OUT_OF_PAGES) == "out of pages"
    assert tg.tg_version() >> 16 == 1


@pytest.mark.parametrize("cfg", [2, 4, 5])
def test_prefill_schedule_bit_exact_on_configs(cfg):
    wl = config(cfg)
    gof = tg.tg_cluster_heads(wl.geom, wl.budget)[1]
    res = tg.tg_reserve(wl.geom, wl.ctx_len, wl.ratio, None, gof, np.zeros(0, np.int32), 0, size_query=True)
    C = wl.chunk_len or 512
    for n_xcd in (8, 3, 1):
        got = tg.tg_prefill_schedule(wl.geom, wl.batch, C, 0, res["kv_len"], n_xcd)
        ref, _ = oracle.prefill_schedule(res["kv_len"], 0, C, wl.geom.gqa, n_xcd)
        assert got.tolist() == ref.tolist()


@settings(max_examples=40, deadline=None)
@given(st.data())
def test_prefill_schedule_random_bit_exact(data):
    H = data.draw(st.sampled_from([1, 2, 4, 8]))
    gqa = data.draw(st.integers(1, 16))
    L = data.draw(st.integers(1, 3))
    B = data.draw(st.integers(1, 5))
    C = data.draw(st.integers(1, 1200))
    n_xcd = data.draw(st.integers(1, 12))
    layer = data.draw(st.integers(0, L - 1))
    rng = np.random.default_rng(data.draw(st.integers(0, 2**31)))
    kv = rng.integers(0, data.draw(st.sampled_from([1, 70, 3000])), size=(B, L, H)).astype(np.int32)
    geom = Geometry(L, H, H * gqa, 128, 16, 1)
    got = tg.tg_prefill_schedule(geom, B, C, layer, kv, n_xcd)
    ref, _ = oracle.prefill_schedule(kv, layer, C, gqa, n_xcd)
    assert got.tolist() == ref.tolist()


def test_prefill_schedule_errors():
    geom = Geometry(1, 2, 4, 128, 16, 1)
    kv = np.ones((1, 1, 2), np.int32)
    for bad in [dict(n_xcd=0), dict(n_xcd=65)]:
        with pytest.raises(tg.TangramError):
            tg.tg_prefill_schedule(geom, 1, 8, 0, kv, **bad)
    with pytest.raises(tg.TangramError):
        tg.tg_prefill_schedule(geom, 1, 0, 0, kv)
    with pytest.raises(tg.TangramError):
        tg.tg_prefill_schedule(geom, 1, 8, 1, kv)


def test_weighted_fill_config3_layer_bit_exact_and_errors():
    wl = config(3)
    gof = tg.tg_cluster_heads(wl.geom, wl.budget)[1]
    need = tg.tg_reserve(wl.geom, wl.ctx_len, wl.ratio, None, gof, np.zeros(0, np.int32), 0, size_query=True)
    pool = pool_pages_for(need["pages_needed"])
    w = np.where((np.arange(1024) // 4) % 8 % 2 == 1, 955, 1044).astype(np.int32)
    _full_compare(wl.geom, wl.batch, wl.ctx_len, wl.ratio, wl.budget, free_list(wl, pool), pool, mode=3,
                  n_bins=1024, split_target=1, layers=[5], bin_weights=w)
    geom = Geometry(1, 2, 4, 128, 16, 1)
    kv = np.full((1, 1, 2), 40, np.int32)
    off = np.array([0, 3, 6], np.int64)
    gof1, sof1 = np.array([[0, 1]], np.int32), np.zeros((1, 2), np.int32)
    for bad, mode in [([0, 1], 3), ([1, 65536], 3), ([1, 1], 0)]:
        with pytest.raises(tg.TangramError):
            tg.tg_build_plan(geom, 1, 0, kv, off, gof1, sof1, mode, 2, 4, bin_weights=np.array(bad, np.int32))
