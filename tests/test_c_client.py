"""The C ABI from plain C: tests/c_abi_client.c is compiled with the system C compiler against
include/tangram.h, linked to libtangram.so and run (host calls only, no GPU, no Python in the path);
its printed results must equal the hand-derived config-1 values in tests/golden/config1_hand.json."""
import json
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2606_06302_amd")
GOLD = json.load(open(os.path.join(ROOT, "tests", "golden", "config1_hand.json")))


@pytest.fixture(scope="module")
def client_output(tmp_path_factory):
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    if not os.path.exists(os.path.join(PKG, "libtangram.so")):
        pytest.fail("libtangram.so is not built (python -m paper_2606_06302_amd.build)")
    exe = tmp_path_factory.mktemp("cabi") / "c_abi_client"
    subprocess.run([cc, "-std=c99", "-Wall", "-Wextra", "-Werror", f"-I{os.path.join(ROOT, 'include')}",
                    os.path.join(ROOT, "tests", "c_abi_client.c"), f"-L{PKG}", "-ltangram", f"-Wl,-rpath,{PKG}",
                    "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout
    return {line.split()[0]: [int(x) for x in line.split()[1:]] for line in out.splitlines() if line.strip()}


def _flat(x):
    return [v for sub in x for v in (_flat(sub) if isinstance(sub, list) else [sub])] if isinstance(x, list) else [x]


def test_clustering_and_reservation(client_output):
    o = client_output
    assert o["perm"] == _flat(GOLD["perm"])
    assert o["group_of"] == _flat(GOLD["group_of"])
    assert o["slot_of"] == _flat(GOLD["slot_of"])
    assert o["kv_len"] == _flat(GOLD["kv_len"])
    assert o["group_len"] == _flat(GOLD["group_len"])
    assert o["offsets"] == GOLD["offsets"]
    assert o["pages_needed"] == [GOLD["pages_needed"]] == o["pages_needed_query"]


def test_split_map_and_plans(client_output):
    o = client_output
    assert o["split_map_ncta256"] == _flat(GOLD["split_map"]["hp2_ncta256"])
    assert o["split_map_ncta8"] == _flat(GOLD["split_map"]["hp2_ncta8"])
    for key, gold in (("plan_aot", GOLD["plan_split_target16_bins8"]), ("plan_fill", GOLD["plan_fill_bins8"])):
        assert o[f"{key}_items"] == _flat(gold["items"]), key
        assert o[f"{key}_bin_offsets"] == gold["bin_offsets"], key
        assert o[f"{key}_unit_splits"] == _flat(gold["unit_splits"]), key
        assert o[f"{key}_num_partials"] == [gold["num_partials"]], key


def test_uniform_and_naive_plans(client_output):
    """The static-split baselines from plain C: UNIFORM at 64 bins and NAIVE, against the hand values."""
    from test_oracle_pins import uniform_gold_items
    o = client_output
    gold = GOLD["plan_uniform_bins64"]
    assert o["plan_uniform_items"] == _flat(uniform_gold_items(gold))
    assert o["plan_uniform_bin_offsets"] == list(range(gold["num_bins"] + 1))
    assert o["plan_uniform_num_bins"] == [gold["num_bins"]]
    assert o["plan_uniform_unit_splits"] == _flat(gold["unit_splits"])
    assert o["plan_uniform_unit_partial_base"] == _flat(gold["unit_partial_base"])
    assert o["plan_uniform_num_partials"] == [gold["num_partials"]]
    gold = GOLD["plan_naive"]
    assert o["plan_naive_items"] == _flat(gold["items"])
    assert o["plan_naive_bin_offsets"] == gold["bin_offsets"]
    assert o["plan_naive_num_bins"] == [gold["num_bins"]]
    assert o["plan_naive_unit_partial_base"] == _flat(gold["unit_partial_base"])
    assert o["plan_naive_num_partials"] == [0]


def test_error_code_and_version(client_output):
    assert client_output["bad_geometry"] == [-1]   # TG_ERR_INVALID_ARG
    assert client_output["version"][0] >> 16 == 1
