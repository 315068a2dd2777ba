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


def test_c_struct_layouts_match_the_binding(tmp_path):
    """Compiles include/tangram.h with the host C compiler and compares sizeof / offsetof of every
    argument struct with the ctypes and numpy layouts the binding uses."""
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        import pytest
        pytest.skip("no host C compiler")
    structs = {"tg_decode_args": tg.tg_decode_args, "tg_prefill_args": tg.tg_prefill_args,
               "tg_compress_args": tg.tg_compress_args, "tg_geometry": tg.tg_geometry,
               "tg_footprint": tg.tg_footprint, "tg_append_args": tg.tg_append_args}
    items = {"tg_work_item": tg.WORK_ITEM_DTYPE, "tg_compress_item": tg.COMPRESS_ITEM_DTYPE}
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "tangram.h"', "int main(void) {"]
    for name, cls in structs.items():
        lines.append(f'printf("{name} %zu\\n", sizeof({name}));')
        for f in cls._fields_:
            lines.append(f'printf("{name}.{f[0]} %zu\\n", offsetof({name}, {f[0]}));')
    for name, dt in items.items():
        lines.append(f'printf("{name} %zu\\n", sizeof({name}));')
        for f in dt.names:
            lines.append(f'printf("{name}.{f} %zu\\n", offsetof({name}, {f}));')
    lines.append('printf("TG_COMPRESS_MAX_CHUNK %d\\nTG_COMPRESS_MAX_ROWS %d\\nTG_COMPRESS_ONE_LAUNCH_MAX_CHUNK %d\\n", '
                 'TG_COMPRESS_MAX_CHUNK, TG_COMPRESS_MAX_ROWS, TG_COMPRESS_ONE_LAUNCH_MAX_CHUNK);')
    lines.append("return 0; }")
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.run([cc, "-std=c99", f"-I{os.path.join(ROOT, 'include')}", str(src), "-o", str(exe)], check=True)
    got = dict(line.split() for line in subprocess.run([str(exe)], capture_output=True, text=True,
                                                       check=True).stdout.splitlines())
    for name, cls in structs.items():
        assert int(got[name]) == ctypes.sizeof(cls), name
        for f in cls._fields_:
            assert int(got[f"{name}.{f[0]}"]) == getattr(cls, f[0]).offset, (name, f[0])
    for name, dt in items.items():
        assert int(got[name]) == dt.itemsize, name
        for f in dt.names:
            assert int(got[f"{name}.{f}"]) == dt.fields[f][1], (name, f)
    assert int(got["TG_COMPRESS_MAX_CHUNK"]) == tg.TG_COMPRESS_MAX_CHUNK
    assert int(got["TG_COMPRESS_MAX_ROWS"]) == tg.TG_COMPRESS_MAX_ROWS
    assert int(got["TG_COMPRESS_ONE_LAUNCH_MAX_CHUNK"]) == tg.TG_COMPRESS_ONE_LAUNCH_MAX_CHUNK
