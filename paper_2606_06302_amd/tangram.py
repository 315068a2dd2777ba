"""ctypes binding of libtangram.so (include/tangram.h), one Python function per C call.

Argument marshalling only: every step of the path runs in the C++/HIP
library.  Host calls take numpy arrays; device calls take torch tensors that
already live on the GPU (their data_ptr() is passed through) and a stream.
If the library has not been built, importing this module raises ImportError
- there is no fallback implementation.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtangram.so")

TG_OK, TG_ERR_INVALID_ARG, TG_ERR_OUT_OF_PAGES, TG_ERR_BUFFER_TOO_SMALL, TG_ERR_UNSUPPORTED, TG_ERR_HIP = 0, -1, -2, -3, -4, -5
TG_ERR_NO_MEMORY = -6
TG_F32, TG_BF16 = 0, 1
TG_GROUP_CLUSTERED, TG_GROUP_ADJACENT = 0, 1
TG_PLAN_AOT, TG_PLAN_NAIVE, TG_PLAN_UNIFORM, TG_PLAN_AOT_FILL, TG_PLAN_SPLIT_MAP = 0, 1, 2, 3, 4
TG_PLAN_OPEN_END = 0x100

# the 32-byte tg_work_item
WORK_ITEM_DTYPE = np.dtype([("pt_base", "<i8"), ("b", "<i4"), ("kv_head", "<i4"), ("slot", "<i4"),
                            ("tok_begin", "<i4"), ("tok_end", "<i4"), ("out_idx", "<i4")])
assert WORK_ITEM_DTYPE.itemsize == 32

# the 40-byte tg_compress_item
COMPRESS_ITEM_DTYPE = np.dtype([("pt_base", "<i8"), ("b", "<i4"), ("kv_head", "<i4"), ("slot", "<i4"),
                                ("n_valid", "<i4"), ("cursor", "<i4"), ("count", "<i4"), ("rank_begin", "<i4"),
                                ("rank_end", "<i4")])
assert COMPRESS_ITEM_DTYPE.itemsize == 40
TG_COMPRESS_MAX_CHUNK, TG_COMPRESS_MAX_ROWS, TG_COMPRESS_ONE_LAUNCH_MAX_CHUNK = 16384, 256, 1024


class TangramError(RuntimeError):
    def __init__(self, code, where, detail):
        super().__init__(f"{where}: {detail} (status {code})")
        self.code = code


class tg_geometry(C.Structure):
    _fields_ = [("num_layers", C.c_int32), ("num_kv_heads", C.c_int32), ("num_q_heads", C.c_int32),
                ("head_dim", C.c_int32), ("page_size", C.c_int32), ("heads_per_group", C.c_int32)]


class tg_decode_args(C.Structure):
    _fields_ = [("geom", tg_geometry), ("batch", C.c_int32), ("dtype", C.c_int32),
                ("q", C.c_void_p), ("kv_pool", C.c_void_p), ("pt_pages", C.c_void_p),
                ("items", C.c_void_p), ("bin_offsets", C.c_void_p), ("n_bins", C.c_int32),
                ("num_items", C.c_int32), ("unit_splits", C.c_void_p), ("unit_partial_base", C.c_void_p),
                ("num_partials", C.c_int32), ("out", C.c_void_p), ("lse", C.c_void_p),
                ("sm_scale", C.c_float), ("workspace", C.c_void_p), ("workspace_bytes", C.c_size_t),
                ("timestamps", C.c_void_p), ("live_len", C.c_void_p), ("layer", C.c_int32),
                ("merge_counters", C.c_void_p), ("append_k", C.c_void_p), ("append_v", C.c_void_p),
                ("append_full", C.c_void_p)]


class tg_prefill_args(C.Structure):
    _fields_ = [("geom", tg_geometry), ("batch", C.c_int32), ("chunk_len", C.c_int32), ("layer", C.c_int32),
                ("dtype", C.c_int32), ("q", C.c_void_p), ("k_new", C.c_void_p), ("v_new", C.c_void_p),
                ("kv_pool", C.c_void_p), ("pt_pages", C.c_void_p), ("pt_offsets", C.c_void_p),
                ("kv_len", C.c_void_p), ("group_of", C.c_void_p), ("slot_of", C.c_void_p),
                ("out", C.c_void_p), ("sm_scale", C.c_float), ("workspace", C.c_void_p),
                ("workspace_bytes", C.c_size_t), ("block_order", C.c_void_p), ("num_blocks", C.c_int32)]


class tg_append_args(C.Structure):
    _fields_ = [("geom", tg_geometry), ("batch", C.c_int32), ("layer", C.c_int32), ("dtype", C.c_int32),
                ("k_tok", C.c_void_p), ("v_tok", C.c_void_p), ("kv_pool", C.c_void_p), ("pt_pages", C.c_void_p),
                ("pt_offsets", C.c_void_p), ("group_of", C.c_void_p), ("slot_of", C.c_void_p),
                ("live_len", C.c_void_p), ("full", C.c_void_p)]


class tg_compress_args(C.Structure):
    _fields_ = [("geom", tg_geometry), ("batch", C.c_int32), ("chunk_len", C.c_int32), ("dtype", C.c_int32),
                ("k_new", C.c_void_p), ("v_new", C.c_void_p), ("scores", C.c_void_p), ("kv_pool", C.c_void_p),
                ("pt_pages", C.c_void_p), ("items", C.c_void_p), ("num_items", C.c_int32),
                ("chunk_tokens", C.c_void_p), ("keep_count", C.c_void_p), ("kept", C.c_void_p)]


class tg_footprint(C.Structure):
    _fields_ = [("full_slots", C.c_int64), ("retained_slots", C.c_int64), ("monolithic_slots", C.c_int64),
                ("ragged_slots", C.c_int64), ("ragged_pages", C.c_int64), ("page_tables", C.c_int64)]


# One HIP runtime per process: torch ships its own libamdhip64 (soname
# libamdhip64.so.7) and loads it by file name, so if libtangram.so were loaded
# first (binding the system copy) torch would bring in a second runtime and
# one of the two would see no device.  Importing torch first makes
# libtangram.so bind to the copy torch uses.
try:
    import torch  # noqa: F401
except ImportError:      # host-only use without torch: the system runtime is fine
    pass

if not os.path.exists(_LIB_PATH):
    raise ImportError(f"{_LIB_PATH} is missing: build it with `python -m paper_2606_06302_amd.build` "
                      "(or __graft_entry__.build()); there is no fallback path")
_lib = C.CDLL(_LIB_PATH)

_P = C.c_void_p
_i32, _i64, _f32, _sz = C.c_int32, C.c_int64, C.c_float, C.c_size_t
_G = C.POINTER(tg_geometry)

_SIGS = {
    "tg_status_string": (C.c_char_p, [_i32]),
    "tg_last_error": (C.c_char_p, []),
    "tg_version": (_i32, []),
    "tg_cluster_heads": (_i32, [_G, _P, _i32, _P, _P, _P]),
    "tg_reserve": (_i32, [_G, _i32, _P, _P, _P, _P, _P, _P, _i64, _i64, _P, _P, _P, _P, _i64, _P]),
    "tg_split_map": (_i32, [_G, _P, _P, _i32, _P]),
    "tg_decode_max_ctas": (_i32, [_G, _i32, _i32, _P]),
    "tg_build_plan": (_i32, [_G, _i32, _i32, _P, _P, _P, _P, _i32, _i32, _i32, _P, _P, _i32, _P, _i32, _P, _P,
                             _P, _P, _P]),
    "tg_decode_workspace_bytes": (_sz, [_G, _i32, _i32]),
    "tg_decode": (_i32, [C.POINTER(tg_decode_args), _P]),
    "tg_decode_noalloc": (_i32, [C.POINTER(tg_decode_args), _P]),
    "tg_append": (_i32, [C.POINTER(tg_append_args), _P]),
    "tg_prefill_workspace_bytes": (_sz, [C.POINTER(tg_prefill_args)]),
    "tg_prefill": (_i32, [C.POINTER(tg_prefill_args), _P]),
    "tg_prefill_schedule": (_i32, [_G, _i32, _i32, _i32, _P, _i32, _P, _i32, _P]),
    "tg_compress_plan": (_i32, [_G, _i32, _i32, _i32, _P, _P, _P, _P, _P, _P, _P, _P, _i32, _P, _i32, _P, _P, _P]),
    "tg_compress": (_i32, [C.POINTER(tg_compress_args), _P]),
    "tg_memory_footprint": (_i32, [_G, _i32, _P, _P, _P, _P, C.POINTER(tg_footprint)]),
    "tg_implicit_ratios": (_i32, [_i32, _i32, _i32, _P, C.c_double, _P, _P]),
    "tg_calibrate_budget": (_i32, [_i32, _i32, _i32, _P, C.c_double, C.c_double, _P]),
    "tg_release_requests": (_i32, [_G, _i32, _P, _P, _P, _P, _i64, _P, _P, _i64, _P, _P, _P]),
    "tg_concat_tables": (_i32, [_G, _i32, _P, _P, _i32, _P, _P, _P, _P]),
    "tg_read_probe": (_i32, [_G, _i32, _P, _P, _P, _i64, _i32, _P, _P]),
}
for _name, (_res, _args) in _SIGS.items():
    _fn = getattr(_lib, _name)
    _fn.restype = _res
    _fn.argtypes = _args

EXPORTED = tuple(_SIGS)


def library_path() -> str:
    return _LIB_PATH


def _geom(g) -> tg_geometry:
    if isinstance(g, tg_geometry):
        return g
    return tg_geometry(g.num_layers, g.num_kv_heads, g.num_q_heads, g.head_dim, g.page_size, g.heads_per_group)


def _ptr(a):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def _check(rc, where):
    if rc != TG_OK:
        raise TangramError(rc, where, _lib.tg_last_error().decode())


def _host(a, dtype):
    return np.ascontiguousarray(np.asarray(a), dtype=dtype)


def tg_status_string(code: int) -> str:
    return _lib.tg_status_string(code).decode()


def tg_last_error() -> str:
    return _lib.tg_last_error().decode()


def tg_version() -> int:
    return _lib.tg_version()


def tg_cluster_heads(geom, budget, grouping=TG_GROUP_CLUSTERED):
    """-> (perm, group_of, slot_of), int32 [L][H] each."""
    g = _geom(geom)
    L, H = g.num_layers, g.num_kv_heads
    b = _host(budget, np.float64).reshape(L, H)
    perm, gof, sof = (np.zeros((L, H), np.int32) for _ in range(3))
    _check(_lib.tg_cluster_heads(C.byref(g), _ptr(b), grouping, _ptr(perm), _ptr(gof), _ptr(sof)), "tg_cluster_heads")
    return perm, gof, sof


def tg_reserve(geom, ctx_len, ratio, budget, group_of, free_pages, pool_pages, size_query=False, headroom=None):
    """-> dict(kv_len [B][L][H], group_len [B][L][G], pt_offsets, pt_pages, pages_needed).  headroom [B]
    reserves room for that many decode tokens per request (None: none)."""
    g = _geom(geom)
    L, H, G = g.num_layers, g.num_kv_heads, g.num_kv_heads // max(1, g.heads_per_group)
    ctx = _host(ctx_len, np.int32)
    B = len(ctx)
    r = None if ratio is None else _host(ratio, np.float64).reshape(B, L, H)
    bud = None if budget is None else _host(budget, np.float64).reshape(L, H)
    gof = _host(group_of, np.int32).reshape(L, H)
    free = _host(free_pages, np.int32)
    kv_len = np.zeros((B, L, H), np.int32)
    group_len = np.zeros((B, L, G), np.int32)
    offsets = np.zeros(B * L * G + 1, np.int64)
    need = C.c_int64(0)
    hr = None if headroom is None else _host(np.broadcast_to(headroom, (B,)), np.int32)
    args = (C.byref(g), B, _ptr(ctx), _ptr(hr), _ptr(r), _ptr(bud), _ptr(gof), _ptr(free), len(free), int(pool_pages),
            _ptr(kv_len), _ptr(group_len), _ptr(offsets))
    rc = _lib.tg_reserve(*args, None, 0, C.byref(need))
    _check(rc, "tg_reserve")
    pages = None
    if not size_query:
        pages = np.empty(max(1, need.value), np.int32)
        rc = _lib.tg_reserve(*args, _ptr(pages), need.value, C.byref(need))
        _check(rc, "tg_reserve")
        pages = pages[: need.value]
    return dict(kv_len=kv_len, group_len=group_len, pt_offsets=offsets, pt_pages=pages, pages_needed=need.value)


def tg_split_map(geom, budget, perm, n_cta):
    g = _geom(geom)
    L, H, G = g.num_layers, g.num_kv_heads, g.num_kv_heads // g.heads_per_group
    S = np.zeros((L, G), np.int32)
    _check(_lib.tg_split_map(C.byref(g), _ptr(_host(budget, np.float64)), _ptr(_host(perm, np.int32)), int(n_cta),
                             _ptr(S)), "tg_split_map")
    return S


def tg_decode_max_ctas(geom, dtype, device=0) -> int:
    g = _geom(geom)
    n = C.c_int32(0)
    _check(_lib.tg_decode_max_ctas(C.byref(g), int(dtype), int(device), C.byref(n)), "tg_decode_max_ctas")
    return n.value


def tg_build_plan(geom, batch, layer, kv_len, pt_offsets, group_of, slot_of, mode=TG_PLAN_AOT, n_bins=1,
                  split_target=1, bin_weights=None):
    """-> dict(items (WORK_ITEM_DTYPE), bin_offsets, unit_splits, unit_partial_base, num_items, num_bins,
    num_partials)."""
    g = _geom(geom)
    H = g.num_kv_heads
    kv = _host(kv_len, np.int32)
    off = _host(pt_offsets, np.int64)
    gof = _host(group_of, np.int32)
    sof = _host(slot_of, np.int32)
    splits = np.zeros((batch, H), np.int32)
    base = np.zeros((batch, H), np.int32)
    ni, nb, npart = C.c_int32(0), C.c_int32(0), C.c_int32(0)
    w = None if bin_weights is None else _host(bin_weights, np.int32)
    head = (C.byref(g), int(batch), int(layer), _ptr(kv), _ptr(off), _ptr(gof), _ptr(sof), int(mode), int(n_bins),
            int(split_target), _ptr(w))
    tail = (_ptr(splits), _ptr(base), C.byref(ni), C.byref(nb), C.byref(npart))
    _check(_lib.tg_build_plan(*head, None, 0, None, 0, *tail), "tg_build_plan")
    items = np.zeros(max(1, ni.value), WORK_ITEM_DTYPE)
    bins = np.zeros(nb.value + 1, np.int32)
    _check(_lib.tg_build_plan(*head, _ptr(items), len(items), _ptr(bins), len(bins), *tail), "tg_build_plan")
    return dict(items=items[: ni.value], bin_offsets=bins, unit_splits=splits, unit_partial_base=base,
                num_items=ni.value, num_bins=nb.value, num_partials=npart.value)


def tg_decode_workspace_bytes(geom, batch, num_partials) -> int:
    return int(_lib.tg_decode_workspace_bytes(C.byref(_geom(geom)), int(batch), int(num_partials)))


def _dptr(t):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        return None
    return C.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def make_decode_args(geom, batch, dtype, q, kv_pool, pt_pages, items, bin_offsets, n_bins, num_items,
                     unit_splits, unit_partial_base, num_partials, out, lse=None, sm_scale=0.0,
                     workspace=None, timestamps=None, live_len=None, layer=0,
                     merge_counters=None, append_k=None, append_v=None, append_full=None) -> tg_decode_args:
    """Packs a tg_decode_args from device tensors (kept alive by the caller); timestamps is an
    int64 device tensor of 2*n_bins entries, or None; live_len an int32 [B][L][H] device tensor of
    current lengths for open-ended plans, or None; merge_counters an int32 [B*H] device tensor of
    zeros for the in-launch merge, or None for the two-launch merge; append_k / append_v the
    step's new token rows [B][H][d] for the in-launch append (with live_len), append_full an
    int32 flag the caller clears."""
    return tg_decode_args(_geom(geom), int(batch), int(dtype), _dptr(q), _dptr(kv_pool), _dptr(pt_pages),
                          _dptr(items), _dptr(bin_offsets), int(n_bins), int(num_items), _dptr(unit_splits),
                          _dptr(unit_partial_base), int(num_partials), _dptr(out), _dptr(lse), float(sm_scale),
                          _dptr(workspace), 0 if workspace is None else workspace.numel() * workspace.element_size(),
                          _dptr(timestamps), _dptr(live_len), int(layer), _dptr(merge_counters),
                          _dptr(append_k), _dptr(append_v), _dptr(append_full))


def tg_decode(args: tg_decode_args, stream=None):
    _check(_lib.tg_decode(C.byref(args), _stream(stream)), "tg_decode")


TG_DECODE_NOALLOC_MAX_BYTES = 16 << 20


def tg_decode_noalloc(args: tg_decode_args, stream=None):
    """tg_decode with the partials in the library's static per-device scratch (args.workspace ignored)."""
    _check(_lib.tg_decode_noalloc(C.byref(args), _stream(stream)), "tg_decode_noalloc")


def make_prefill_args(geom, batch, chunk_len, layer, dtype, q, k_new, v_new, kv_pool, pt_pages, pt_offsets,
                      kv_len, group_of, slot_of, out, sm_scale=0.0, workspace=None,
                      block_order=None) -> tg_prefill_args:
    """Packs a tg_prefill_args from device tensors (kept alive by the caller); block_order is the
    device copy of a tg_prefill_schedule result, or None for the default block mapping."""
    return tg_prefill_args(_geom(geom), int(batch), int(chunk_len), int(layer), int(dtype), _dptr(q),
                           _dptr(k_new), _dptr(v_new), _dptr(kv_pool), _dptr(pt_pages), _dptr(pt_offsets),
                           _dptr(kv_len), _dptr(group_of), _dptr(slot_of), _dptr(out), float(sm_scale),
                           _dptr(workspace), 0 if workspace is None else workspace.numel() * workspace.element_size(),
                           _dptr(block_order), 0 if block_order is None else int(block_order.numel()))


def tg_prefill_schedule(geom, batch, chunk_len, layer, kv_len, n_xcd=8):
    """-> int32 array: block k runs (unit, row tile) = divmod(order[k], row_tiles), or nothing if -1."""
    g = _geom(geom)
    kv = _host(kv_len, np.int32)
    n = C.c_int32(0)
    head = (C.byref(g), int(batch), int(chunk_len), int(layer), _ptr(kv), int(n_xcd))
    _check(_lib.tg_prefill_schedule(*head, None, 0, C.byref(n)), "tg_prefill_schedule")
    order = np.zeros(max(1, n.value), np.int32)
    _check(_lib.tg_prefill_schedule(*head, _ptr(order), len(order), C.byref(n)), "tg_prefill_schedule")
    return order[: n.value]


def tg_prefill_workspace_bytes(args: tg_prefill_args) -> int:
    return int(_lib.tg_prefill_workspace_bytes(C.byref(args)))


def tg_prefill(args: tg_prefill_args, stream=None):
    _check(_lib.tg_prefill(C.byref(args), _stream(stream)), "tg_prefill")


def tg_compress_plan(geom, batch, layer, chunk_len, chunk_start, chunk_tokens, ratio, budget, kv_len, pt_offsets,
                     group_of, slot_of, rows_per_item=64):
    """-> dict(items (COMPRESS_ITEM_DTYPE), num_items, keep_count [B][H], write_begin [B][H])."""
    g = _geom(geom)
    H = g.num_kv_heads
    cs = _host(chunk_start, np.int32)
    ct = _host(chunk_tokens, np.int32)
    r = None if ratio is None else _host(ratio, np.float64)
    bud = None if budget is None else _host(budget, np.float64)
    kv = _host(kv_len, np.int32)
    off = _host(pt_offsets, np.int64)
    gof = _host(group_of, np.int32)
    sof = _host(slot_of, np.int32)
    cnt = np.zeros((batch, H), np.int32)
    wb = np.zeros((batch, H), np.int32)
    ni = C.c_int32(0)
    head = (C.byref(g), int(batch), int(layer), int(chunk_len), _ptr(cs), _ptr(ct), _ptr(r), _ptr(bud), _ptr(kv),
            _ptr(off), _ptr(gof), _ptr(sof), int(rows_per_item))
    _check(_lib.tg_compress_plan(*head, None, 0, _ptr(cnt), _ptr(wb), C.byref(ni)), "tg_compress_plan")
    items = np.zeros(max(1, ni.value), COMPRESS_ITEM_DTYPE)
    _check(_lib.tg_compress_plan(*head, _ptr(items), len(items), _ptr(cnt), _ptr(wb), C.byref(ni)),
           "tg_compress_plan")
    return dict(items=items[: ni.value], num_items=ni.value, keep_count=cnt, write_begin=wb)


def make_compress_args(geom, batch, chunk_len, dtype, k_new, v_new, scores, kv_pool, pt_pages, items, num_items,
                       chunk_tokens, keep_count, kept) -> tg_compress_args:
    """Packs a tg_compress_args from device tensors (kept alive by the caller)."""
    return tg_compress_args(_geom(geom), int(batch), int(chunk_len), int(dtype), _dptr(k_new), _dptr(v_new),
                            _dptr(scores), _dptr(kv_pool), _dptr(pt_pages), _dptr(items), int(num_items),
                            _dptr(chunk_tokens), _dptr(keep_count), _dptr(kept))


def tg_compress(args: tg_compress_args, stream=None):
    _check(_lib.tg_compress(C.byref(args), _stream(stream)), "tg_compress")


def tg_memory_footprint(geom, ctx_len, ratio, budget, group_of) -> dict:
    """-> dict of slot counts (full, retained, monolithic, ragged), ragged_pages and page_tables."""
    g = _geom(geom)
    ctx = _host(ctx_len, np.int32)
    r = None if ratio is None else _host(ratio, np.float64)
    bud = None if budget is None else _host(budget, np.float64)
    out = tg_footprint()
    _check(_lib.tg_memory_footprint(C.byref(g), len(ctx), _ptr(ctx), _ptr(r), _ptr(bud),
                                    _ptr(_host(group_of, np.int32)), C.byref(out)), "tg_memory_footprint")
    return {f[0]: int(getattr(out, f[0])) for f in tg_footprint._fields_}


def make_append_args(geom, batch, layer, dtype, k_tok, v_tok, kv_pool, pt_pages, pt_offsets, group_of, slot_of,
                     live_len, full=None) -> tg_append_args:
    """Packs a tg_append_args from device tensors (kept alive by the caller)."""
    return tg_append_args(_geom(geom), int(batch), int(layer), int(dtype), _dptr(k_tok), _dptr(v_tok),
                          _dptr(kv_pool), _dptr(pt_pages), _dptr(pt_offsets), _dptr(group_of), _dptr(slot_of),
                          _dptr(live_len), _dptr(full))


def tg_append(args: tg_append_args, stream=None):
    _check(_lib.tg_append(C.byref(args), _stream(stream)), "tg_append")


def tg_implicit_ratios(scores, rho):
    """scores [L][H][N] float32 -> (ratios [L][H] float64, counts [L][H] int32)."""
    sc = _host(scores, np.float32)
    L, H, N = sc.shape
    r = np.zeros((L, H), np.float64)
    c = np.zeros((L, H), np.int32)
    _check(_lib.tg_implicit_ratios(L, H, N, _ptr(sc), float(rho), _ptr(r), _ptr(c)), "tg_implicit_ratios")
    return r, c


def tg_calibrate_budget(ratios, alpha=2.0, floor=1e-3):
    """ratios [S][L][H] float64 -> budgets [L][H]."""
    r = _host(ratios, np.float64)
    S, L, H = r.shape
    out = np.zeros((L, H), np.float64)
    _check(_lib.tg_calibrate_budget(S, L, H, _ptr(r), float(alpha), float(floor), _ptr(out)), "tg_calibrate_budget")
    return out


def tg_release_requests(geom, pt_offsets, pt_pages, finished):
    """-> (freed page ids, new_offsets, new_pages) for the requests that did not finish."""
    g = _geom(geom)
    off = _host(pt_offsets, np.int64)
    pages = _host(pt_pages, np.int32)
    fin = _host(finished, np.uint8)
    B = len(fin)
    nf, nk, ns = C.c_int64(0), C.c_int64(0), C.c_int32(0)
    head = (C.byref(g), B, _ptr(off), _ptr(pages), _ptr(fin))
    _check(_lib.tg_release_requests(*head, None, 0, None, None, 0, C.byref(nf), C.byref(nk), C.byref(ns)),
           "tg_release_requests")
    per = g.num_layers * (g.num_kv_heads // g.heads_per_group)
    freed = np.zeros(max(1, nf.value), np.int32)
    new_pages = np.zeros(max(1, nk.value), np.int32)
    new_off = np.zeros(ns.value * per + 1, np.int64)
    _check(_lib.tg_release_requests(*head, _ptr(freed), len(freed), _ptr(new_off), _ptr(new_pages), len(new_pages),
                                    C.byref(nf), C.byref(nk), C.byref(ns)), "tg_release_requests")
    return freed[: nf.value], new_off, new_pages[: nk.value]


def tg_concat_tables(geom, offsets_a, pages_a, offsets_b, pages_b):
    """-> (offsets, pages) of batch a followed by batch b."""
    g = _geom(geom)
    per = g.num_layers * (g.num_kv_heads // g.heads_per_group)
    oa, ob = _host(offsets_a, np.int64), _host(offsets_b, np.int64)
    pa, pb = _host(pages_a, np.int32), _host(pages_b, np.int32)
    ba, bb = (len(oa) - 1) // per, (len(ob) - 1) // per
    off = np.zeros((ba + bb) * per + 1, np.int64)
    pages = np.zeros(max(1, int(oa[-1] + ob[-1])), np.int32)
    _check(_lib.tg_concat_tables(C.byref(g), ba, _ptr(oa), _ptr(pa), bb, _ptr(ob), _ptr(pb), _ptr(off), _ptr(pages)),
           "tg_concat_tables")
    return off, pages[: int(oa[-1] + ob[-1])]


def tg_read_probe(geom, dtype, kv_pool, page_ids, slots, n_workers, out, stream=None):
    """Streams the K and V slabs of every (page_ids[i], slots[i]) (device int32 tensors); out is a device
    uint32/int32 tensor of n_workers checksums."""
    _check(_lib.tg_read_probe(C.byref(_geom(geom)), int(dtype), _dptr(kv_pool), _dptr(page_ids), _dptr(slots),
                              int(page_ids.numel()), int(n_workers), _dptr(out), _stream(stream)), "tg_read_probe")
