"""Integer rows on the GPU record: page tables and partition plans built by the oracle drive the kernels.

For every case the oracle's clustering (Section 4.2.2), reservation (Eq. 4, Sections 4.1 and 4.2.1), split map
(Algorithm 1) and partition plan of every mode are computed on the host.  The library's tg_cluster_heads,
tg_reserve, tg_split_map and tg_build_plan must equal them bit for bit.  Then the oracle's own tables and plans,
packed into the C structs, are uploaded and tg_decode runs from them; its outputs must match the oracle's attention
within the dtype tolerance.  So a GPU run alone checks the whole path from budgets to outputs.
"""
import types

import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import check_close, retained_mask, say
from workloads import Geometry, config, custom, free_list, host_pool, host_q_decode, pool_pages_for

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from paper_2606_06302_amd import tangram as tg
    from paper_2606_06302_amd.device import bind_decode, to_device, upload_plan

MODES = {"aot": oracle.MODE_AOT, "naive": oracle.MODE_NAIVE, "uniform": oracle.MODE_UNIFORM,
         "fill": oracle.MODE_FILL, "splitmap": oracle.MODE_SPLIT_MAP}


def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _as_c_plan(plan, n_units_shape):
    """The oracle's plan in the layout tg_build_plan writes (32-byte items, int32 arrays)."""
    items = np.zeros(max(1, len(plan["items"])), tg.WORK_ITEM_DTYPE)
    for i, it in enumerate(plan["items"]):
        items[i] = it
    return dict(items=items[: len(plan["items"])], num_items=len(plan["items"]),
                bin_offsets=np.asarray(plan["bin_offsets"], np.int32), num_bins=len(plan["bin_offsets"]) - 1,
                unit_splits=np.asarray(plan["unit_splits"], np.int32).reshape(n_units_shape),
                unit_partial_base=np.asarray(plan["unit_partial_base"], np.int32).reshape(n_units_shape),
                num_partials=int(plan["num_partials"]))


def _items(p):
    return [tuple(int(x) for x in it) for it in p["items"]]


@pytest.mark.parametrize("case", ["config1", "bf16-gqa8", "f32-gqa3-hp1", "bf16-gqa5-hp4"])
def test_oracle_tables_and_plans_drive_the_decode(case):
    _gpu()
    if case == "config1":
        wl = config(1)
    elif case == "bf16-gqa8":
        wl = custom(9101, Geometry(2, 8, 64, 128, 16, 2), 3, "bf16", (100, 3000), kv_scale=0.5)
    elif case == "f32-gqa3-hp1":
        wl = custom(9102, Geometry(2, 4, 12, 64, 16, 1), 2, "f32", (30, 900))
    else:
        wl = custom(9103, Geometry(1, 8, 40, 128, 16, 4), 4, "bf16", (16, 2500), kv_scale=0.5)
    g = wl.geom
    L, H, G, P, B = g.num_layers, g.num_kv_heads, g.num_groups, g.page_size, wl.batch
    say(f"oracle tables {case}: B={B} L={L} H={H} Hq={g.num_q_heads} d={g.head_dim} Hp={g.heads_per_group} "
        f"ctx={wl.ctx_len.tolist()}")

    # integer rows a1-a5 on the oracle, and the library's results bit for bit
    perm, group_of, slot_of = oracle.cluster_heads(wl.budget, g.heads_per_group)
    lib_perm, lib_gof, lib_sof = tg.tg_cluster_heads(g, wl.budget)
    assert np.array_equal(lib_perm, perm) and np.array_equal(lib_gof, group_of) and np.array_equal(lib_sof, slot_of)
    need = oracle.reserve(wl.ratio, wl.ctx_len, group_of, G, P, np.arange(10**7))["pages_needed"]
    pool_pages = pool_pages_for(need)
    free = free_list(wl, pool_pages)
    res = oracle.reserve(wl.ratio, wl.ctx_len, group_of, G, P, free)
    lib = tg.tg_reserve(g, wl.ctx_len, wl.ratio, None, lib_gof, free, pool_pages)
    assert np.array_equal(lib["kv_len"], res["kv_len"]) and np.array_equal(lib["group_len"], res["group_len"])
    assert np.array_equal(lib["pt_offsets"], res["offsets"]) and np.array_equal(lib["pt_pages"], res["pages"])
    assert lib["pages_needed"] == res["pages_needed"]

    # device inputs: NaN in every pool row that holds no retained entry
    tables = types.SimpleNamespace(kv_len=res["kv_len"], pt_offsets=res["offsets"], pt_pages=res["pages"],
                                   group_of=group_of, slot_of=slot_of, pool_pages=pool_pages)
    pool_h = host_pool(wl, pool_pages).reshape(pool_pages, 2, g.heads_per_group, P, g.head_dim)
    pool_h[~retained_mask(tables, wl)] = np.nan
    dt = {"f32": torch.float32, "bf16": torch.bfloat16}[wl.dtype]
    tg_dt = {"f32": tg.TG_F32, "bf16": tg.TG_BF16}[wl.dtype]
    pool = torch.from_numpy(pool_h).to(dt).cuda()
    q = torch.from_numpy(host_q_decode(wl)).to(dt).cuda()
    d_pages = to_device(res["pages"].astype(np.int32), "cuda")
    f64 = lambda t: t.float().cpu().numpy().astype(np.float64)
    pool64, q64 = f64(pool), f64(q)

    n_cta = 48
    S = oracle.split_map(wl.budget, perm, g.heads_per_group, n_cta)
    assert np.array_equal(tg.tg_split_map(g, wl.budget, lib_perm, n_cta), S)
    for name, mode in MODES.items():
        for l in range(L):
            kw = dict(n_bins=n_cta, split_target=3 * n_cta)
            if mode == oracle.MODE_SPLIT_MAP:
                kw["bin_weights"] = S[l]
            plan = oracle.partition_plan(res["kv_len"], res["offsets"], group_of, slot_of, l, num_layers=L,
                                         num_groups=G, page_size=P, mode=mode, **kw)
            lp = tg.tg_build_plan(g, B, l, lib["kv_len"], lib["pt_offsets"], lib_gof, lib_sof, mode, kw["n_bins"],
                                  kw["split_target"], bin_weights=kw.get("bin_weights"))
            cp = _as_c_plan(plan, (B, H))
            assert _items(lp) == _items(cp), (name, l)
            assert np.array_equal(lp["bin_offsets"], cp["bin_offsets"]), (name, l)
            assert np.array_equal(lp["unit_splits"], cp["unit_splits"]), (name, l)
            assert np.array_equal(lp["unit_partial_base"], cp["unit_partial_base"]), (name, l)
            assert lp["num_partials"] == cp["num_partials"], (name, l)

            # the decode runs from the oracle's plan and tables
            out = torch.full((B, g.num_q_heads, g.head_dim), float("nan"), dtype=dt, device="cuda")
            lse = torch.full((B, g.num_q_heads), float("nan"), dtype=torch.float32, device="cuda")
            dp = upload_plan(g, B, cp, "cuda")
            bind_decode(dp, g, B, tg_dt, q[l], pool, d_pages, out, lse)
            tg.tg_decode(dp.args)
            torch.cuda.synchronize()
            O, lse_ref = oracle.decode_attention(q64[l], pool64, l, geom=g, batch=B, kv_len=res["kv_len"],
                                                 offsets=res["offsets"], pages=res["pages"], group_of=group_of,
                                                 slot_of=slot_of)
            check_close(f64(out).reshape(-1, g.head_dim), O.reshape(-1, g.head_dim), wl.dtype,
                        f"{case} {name} layer {l}")
            err = float(np.abs(lse.cpu().numpy() - lse_ref).max())
            assert err <= (1e-4 if wl.dtype == "f32" else 2e-3), (case, name, l, err)
        say(f"  {name}: {cp['num_items']} items, {cp['num_bins']} bins, {cp['num_partials']} partials ok")
