"""tg_decode_noalloc: the decode with its split partials in the library's static per-device scratch.

Checked against tg_decode (same plan, same inputs, the partials in a caller workspace) and against the fp64
oracle, on two calls in a row, the second with a smaller input, for the MFMA kernel (bf16, d 128) and the generic
kernel (fp32, d 64); plus the host-side size limit.
"""
import numpy as np
import pytest
import torch

from gpu_helpers import compare_layer, poisoned_host_pool, say
from workloads import Geometry, custom

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from paper_2606_06302_amd import tangram as tg
    from paper_2606_06302_amd.runner import DecodeSession, Tables


def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _session(wl, mode, n_bins, fused=False):
    tables = Tables(wl)
    dt = {"f32": torch.float32, "bf16": torch.bfloat16}[wl.dtype]
    pool = torch.from_numpy(poisoned_host_pool(wl, tables)).to(dt).cuda()
    return DecodeSession(wl, tables=tables, mode=mode, n_bins=n_bins, split_target=2 * n_bins, fill="host",
                         pool=pool, fused_merge=fused)


@pytest.mark.parametrize("dtype,d,gqa,fused", [("bf16", 128, 8, False), ("f32", 64, 3, False), ("bf16", 128, 8, True)])
def test_noalloc_matches_workspace_decode_twice(dtype, d, gqa, fused):
    _gpu()
    big = custom(8801 + d, Geometry(2, 8, 8 * gqa, d, 16, 2), 6, dtype, (300, 6000), kv_scale=0.5)
    small = custom(8802 + d, Geometry(1, 4, 4 * gqa, d, 16, 2), 2, dtype, (20, 900), kv_scale=0.5)
    for wl, n_bins in ((big, 160), (small, 24)):          # the second call: a smaller input
        s = _session(wl, tg.TG_PLAN_AOT_FILL, n_bins, fused)
        parts = [s.plans[l]["num_partials"] for l in s.layers]
        say(f"noalloc {dtype} d{d} gqa{gqa}: B={wl.batch} L={wl.geom.num_layers} partials {parts}")
        assert max(parts) > 0
        s.run_step()
        torch.cuda.synchronize()
        ref_out, ref_lse = s.out.clone(), s.lse.clone()
        s.out.fill_(float("nan"))
        s.lse.fill_(float("nan"))
        torch.cuda.synchronize()
        for l in s.layers:
            tg.tg_decode_noalloc(s.dplans[l].args)
        torch.cuda.synchronize()
        assert torch.equal(s.out, ref_out) and torch.equal(s.lse, ref_lse)
        for l in s.layers:
            compare_layer(s, l, what=f"noalloc {dtype} layer {l}")


def test_noalloc_size_limit_is_checked_on_the_host():
    _gpu()
    g = Geometry(1, 8, 64, 128, 16, 2)
    per_partial = tg.tg_decode_workspace_bytes(g, 1, 1000) / 1000
    too_many = int(tg.TG_DECODE_NOALLOC_MAX_BYTES / per_partial) + 8
    assert tg.tg_decode_workspace_bytes(g, 1, too_many) > tg.TG_DECODE_NOALLOC_MAX_BYTES
    args = tg.tg_decode_args(tg._geom(g), 4, tg.TG_BF16, None, None, None, None, None, 16, 1, None, None, too_many,
                             None, None, 0.0, None, 0, None, None, 0)
    with pytest.raises(tg.TangramError) as e:
        tg.tg_decode_noalloc(args)
    assert e.value.code == tg.TG_ERR_BUFFER_TOO_SMALL
    assert "scratch" in tg.tg_last_error()
