"""The Chrome-trace export (argus_attr_chrome_trace, host code): the JSON
parses, and every drawn slice is checked against the instances and probe
groups it was made from -- lane, start, duration and nesting of the
percentile bands (the lane layout of the paper's Appendix B)."""
from __future__ import annotations

import json
import os

import numpy as np
import pytest

from golden_util import random_malformed, records_from_rows

B, E = 1, 2


@pytest.fixture(scope="module")
def lib():
    from paper_2609_12299_amd import attr
    if not os.path.exists(attr.LIB_PATH):
        from paper_2609_12299_amd import build
        build.build()
    return attr


def _export(lib, tmp_path, inst, R, cpu, shift, groups=None, mean=None, names=None, unmatched=False):
    path = str(tmp_path / "trace.json")
    rc = lib.argus_attr_chrome_trace(inst, path, R, cpu, shift, groups, mean, names, unmatched)
    assert rc == 0
    with open(path) as f:
        return json.load(f)


def test_reference_and_probe_lanes(lib, oracle_mod, tmp_path):
    # ctx 5 (group 1 with shift 2, local warp 1): region 0 around two loads
    # (region 1); ctx 4 one mismatched pair
    rows = [(1000, 5, 0, B), (1100, 5, 1, B), (1300, 5, 1, E), (1400, 5, 1, B), (1450, 5, 1, E),
            (2000, 5, 0, E), (0, 4, 0, B), (10, 4, 1, E)]
    o = oracle_mod.run(records_from_rows(rows), 2)
    inst = o["instances"]
    import oracle
    pr = np.zeros(5, oracle.PROBE_DTYPE)
    for i, d in enumerate((40, 10, 30, 20, 50)):
        pr[i] = (0, d, 5, 0, 1, 0, 0)
    p = oracle_mod.probes(inst, 2, pr)
    t = _export(lib, tmp_path, inst, 2, 100.0, 2, p["groups"], p["mean"], ["main", "load \"A\""])
    ev = t["traceEvents"]
    ref = [e for e in ev if e.get("cat") == "reference"]
    assert len(ref) == 3  # the mismatched pair of ctx 4 is left out
    by_inst = {e["args"]["instance"]: e for e in ref}
    for x, e in by_inst.items():
        a = inst[x]
        assert e["pid"] == int(a["ctx_key"]) >> 2
        assert e["tid"] == (int(a["ctx_key"]) & 3) * 1024 + int(a["level"])
        assert e["ts"] == pytest.approx(int(a["t_begin"]) / 100.0, abs=1e-4)
        assert e["dur"] == pytest.approx((int(a["t_end"]) - int(a["t_begin"])) / 100.0, abs=1e-4)
    assert by_inst[1]["name"] == "main" and by_inst[2]["name"] == 'load "A"'
    mean = [e for e in ev if e.get("cat") == "mean"]
    assert len(mean) == 1 and mean[0]["ts"] == pytest.approx(11.0) and mean[0]["dur"] == pytest.approx(0.3)
    bands = [e for e in ev if e.get("cat") == "percentile"]
    assert [e["name"].split()[-1] for e in bands] == ["p80", "p60", "p40", "p20", "p0"]
    assert [round(e["dur"] * 100) for e in bands] == [40, 30, 20, 10, 10]
    assert all(e["tid"] == mean[0]["tid"] + 1 == 1024 + 8 + 1 for e in bands)
    names = {(e["pid"], e["tid"]): e["args"]["name"] for e in ev if e.get("name") == "thread_name"}
    used = {(e["pid"], e["tid"]) for e in ev if e["ph"] == "X"}
    assert used == set(names)
    t2 = _export(lib, tmp_path, inst, 2, 100.0, 2, unmatched=True)
    assert sum(1 for e in t2["traceEvents"] if e.get("cat") == "reference") == 4


def test_random_trace_roundtrip(lib, oracle_mod, tmp_path):
    rng = np.random.default_rng(31)
    R = 5
    inst = oracle_mod.run(random_malformed(rng, 3000, 6, R, 100000), R)["instances"]
    t = _export(lib, tmp_path, inst, R, 1755.0, 1)
    ref = [e for e in t["traceEvents"] if e.get("cat") == "reference"]
    matched = (inst["end_region_id"] != 0xFFFF) & (inst["end_region_id"] == inst["region_id"])
    assert sorted(e["args"]["instance"] for e in ref) == np.nonzero(matched)[0].tolist()
    for e in ref:
        a = inst[e["args"]["instance"]]
        assert e["args"]["cycles"] == int(a["t_end"]) - int(a["t_begin"])
        assert e["tid"] % 1024 == min(int(a["level"]), 7)


def test_export_errors(lib, oracle_mod, tmp_path):
    inst = oracle_mod.run(records_from_rows([(0, 0, 0, B), (5, 0, 0, E)]), 1)["instances"]
    assert lib.argus_attr_chrome_trace(inst, str(tmp_path / "x.json"), 1, 0.0) == -1
    assert lib.argus_attr_chrome_trace(inst, str(tmp_path / "x.json"), 0, 1.0) == -1
    bad = np.zeros((1, 10), np.uint64)
    bad[0, 0] = 7  # names an instance that does not exist
    assert lib.argus_attr_chrome_trace(inst, str(tmp_path / "x.json"), 1, 1.0, 0, bad,
                                       np.zeros(1)) == -1
    assert lib.argus_attr_chrome_trace(inst, str(tmp_path / "no" / "dir" / "x.json"), 1, 1.0) == -7
