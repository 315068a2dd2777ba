"""The C-ABI library loads and exports every function include/tangram.h declares (CPU only)."""
import ctypes
import os
import re

from paper_2606_06302_amd import tangram as tg

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    names = set()
    for fn in os.listdir(os.path.join(ROOT, "include")):
        if fn.endswith(".h"):
            text = open(os.path.join(ROOT, "include", fn)).read()
            text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
            names |= set(re.findall(r"^\s*(?:const\s+)?[A-Za-z_][A-Za-z0-9_]*\s*\*?\s*(tg_[a-z0-9_]+)\s*\(", text, re.M))
    return names


def test_every_declared_symbol_is_exported():
    declared = declared_functions()
    assert {"tg_reserve", "tg_build_plan", "tg_decode", "tg_prefill", "tg_split_map", "tg_cluster_heads"} <= declared
    lib = ctypes.CDLL(tg.library_path())
    missing = [n for n in sorted(declared) if not hasattr(lib, n)]
    assert not missing, missing
    assert declared == set(tg.EXPORTED), declared ^ set(tg.EXPORTED)


def test_struct_sizes_match_header():
    assert ctypes.sizeof(tg.tg_geometry) == 24
    assert tg.WORK_ITEM_DTYPE.itemsize == 32
    # tg_decode_args / tg_prefill_args are plain C structs of the declared field order
    assert [f[0] for f in tg.tg_decode_args._fields_][:4] == ["geom", "batch", "dtype", "q"]
