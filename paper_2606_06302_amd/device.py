"""Device-memory plumbing around the C ABI (torch owns allocations and streams).

Nothing here computes any part of the method: it uploads the host tables that
tg_reserve / tg_build_plan produced and packs tg_decode_args once per layer so
a timed loop only enqueues tg_decode calls.
"""
from __future__ import annotations

import dataclasses

import numpy as np
import torch

from . import tangram as tg


def to_device(a: np.ndarray, device) -> torch.Tensor:
    a = np.ascontiguousarray(a)
    if a.dtype.fields is not None:          # structured (work items): raw bytes
        a = a.view(np.uint8)
    return torch.from_numpy(a).to(device)


@dataclasses.dataclass
class DevicePlan:
    """One layer's partition plan in device memory plus its packed decode args."""
    host: dict
    items: torch.Tensor
    bin_offsets: torch.Tensor
    unit_splits: torch.Tensor
    unit_partial_base: torch.Tensor
    workspace: torch.Tensor
    args: tg.tg_decode_args = None

    @property
    def n_bins(self):
        return self.host["num_bins"]


def upload_plan(geom, batch, plan: dict, device) -> DevicePlan:
    ws_bytes = tg.tg_decode_workspace_bytes(geom, batch, plan["num_partials"])
    return DevicePlan(
        host=plan,
        items=to_device(plan["items"] if plan["num_items"] else np.zeros(1, tg.WORK_ITEM_DTYPE), device),
        bin_offsets=to_device(plan["bin_offsets"], device),
        unit_splits=to_device(plan["unit_splits"], device),
        unit_partial_base=to_device(plan["unit_partial_base"], device),
        workspace=torch.empty(max(256, ws_bytes), dtype=torch.uint8, device=device),
    )


def bind_decode(dp: DevicePlan, geom, batch, dtype, q, kv_pool, pt_pages, out, lse=None, sm_scale=0.0,
                live_len=None, layer=0, merge_counters=None):
    """Packs (and stores on dp) the tg_decode_args for this layer; merge_counters (int32 [B*H] zeros,
    shared by calls on one stream) selects the in-launch merge."""
    dp.args = tg.make_decode_args(geom, batch, dtype, q, kv_pool, pt_pages, dp.items, dp.bin_offsets,
                                  dp.host["num_bins"], dp.host["num_items"], dp.unit_splits,
                                  dp.unit_partial_base, dp.host["num_partials"], out, lse, sm_scale,
                                  dp.workspace, live_len=live_len, layer=layer, merge_counters=merge_counters)
    return dp.args
