"""Parity at the full workload sizes, in the launch configuration the benchmark
times (instances and exclusive times written, default sort path).

* The four smaller workloads (2^16 .. 2^26 records) are compared whole with
  the oracle, bit for bit.
* The 2^28-record trace (4 GiB) is run whole on the GPU and compared whole
  with the oracle, bit for bit, after cheap checks of properties that hold at
  any size (counter identities, per-region statistics recomputed from the
  instance array).
"""
from __future__ import annotations

import numpy as np
import pytest

from golden_util import RECORD_DTYPE, RS_FIELDS
from gpu_util import assert_parity, gpu_run, log, oracle_run

pytestmark = pytest.mark.gpu

U64_MAX = np.uint64(0xFFFFFFFFFFFFFFFF)
NO_PARENT = 0xFFFFFFFF
NO_END = 0xFFFF


def _params(d):
    return {k: d[k] for k in ("num_regions", "num_classes", "region_class", "group_shift", "num_groups")}


@pytest.mark.parametrize("cfg", [1, 2, 4, 3])
def test_full_size_whole(oracle_mod, tracegen_mod, cfg):
    d = tracegen_mod.generate(cfg, threads=16)
    p = _params(d)
    log(f"[gpu] full-size config {cfg}: n={len(d['records'])}")
    assert_parity(gpu_run(d["records"], p), oracle_run(oracle_mod, d["records"], p),
                  what=f"full cfg{cfg}")


def _bit_width(x: np.ndarray) -> np.ndarray:
    """Number of significant bits of each u64 (0 for 0), exactly."""
    x = x.astype(np.uint64)
    bw = np.zeros(x.shape, np.int64)
    for s in (32, 16, 8, 4, 2, 1):
        big = (x >> np.uint64(s)) != 0
        bw += np.where(big, s, 0)
        x = np.where(big, x >> np.uint64(s), x)
    return bw + (x != 0)


def _region_stats_from_instances(inst: np.ndarray, excl: np.ndarray, R: int) -> dict:
    """Per-region statistics of the matched instances, from the instance array."""
    closed = inst["end_region_id"] != NO_END
    matched = closed & (inst["end_region_id"] == inst["region_id"])
    reg = inst["region_id"][matched].astype(np.int64)
    d = (inst["t_end"][matched] - inst["t_begin"][matched]).astype(np.uint64)
    e = excl[matched].astype(np.uint64)
    out = {}
    out["count"] = np.bincount(reg, minlength=R).astype(np.uint64)
    # u64 sums that wrap: split into 32-bit halves, sum exactly in u64 per half
    for name, v in (("incl_sum", d), ("excl_sum", e)):
        lo = np.zeros(R, np.uint64)
        hi = np.zeros(R, np.uint64)
        np.add.at(lo, reg, v & np.uint64(0xFFFFFFFF))
        np.add.at(hi, reg, v >> np.uint64(32))
        out[name] = lo + (hi << np.uint64(32))
    for name, v, fn, init in (("incl_min", d, np.minimum, U64_MAX), ("incl_max", d, np.maximum, 0),
                              ("excl_min", e, np.minimum, U64_MAX), ("excl_max", e, np.maximum, 0)):
        a = np.full(R, init, np.uint64)
        fn.at(a, reg, v)
        out[name] = a
    for name, v in (("hist_incl", d), ("hist_excl", e)):
        h = np.zeros(R * 65, np.uint64)
        np.add.at(h, reg * 65 + _bit_width(v), 1)
        out[name] = h.reshape(R, 65)
    # ambiguity counts that the instance array determines
    unc = ~closed
    out["unclosed"] = np.bincount(inst["region_id"][unc].astype(np.int64), minlength=R).astype(np.uint64)
    mism = closed & ~matched
    out["mism_as_begin"] = np.bincount(inst["region_id"][mism].astype(np.int64), minlength=R).astype(np.uint64)
    out["mism_as_end"] = np.bincount(inst["end_region_id"][mism].astype(np.int64), minlength=R).astype(np.uint64)
    par = inst["parent"]
    has_par = matched & (par != NO_PARENT)
    idx = np.nonzero(has_par)[0]
    selfn = idx[inst["region_id"][par[idx]] == inst["region_id"][idx]]
    out["self_nested"] = np.bincount(inst["region_id"][selfn].astype(np.int64), minlength=R).astype(np.uint64)
    return out


def test_run_lists_in_several_bursts(oracle_mod):
    """2^25 records of 4096 contexts interleaved 8 at a time: 32 runs per
    256-record chunk, so every ingest wave stages more runs than its buffer
    holds and writes its run list out in several bursts, while the context
    sort over runs is still taken.  Compared whole with the oracle."""
    rng = np.random.default_rng(25)
    C, per, step = 4096, 8192, 8
    n = C * per
    # per context, groups of four: BEGIN r1, BEGIN r2, END r2, END r1
    r1 = rng.integers(0, 6, size=(C, per // 4))
    r2 = rng.integers(0, 6, size=(C, per // 4))
    region = np.stack([r1, r2, r2, r1], axis=2).reshape(C, per)
    kind = np.tile(np.array([1, 1, 2, 2], np.uint8), per // 4)[None, :].repeat(C, axis=0)
    ts = np.cumsum(rng.integers(1, 50, size=(C, per), dtype=np.uint64), axis=1, dtype=np.uint64)
    ts += rng.integers(0, 1 << 30, size=(C, 1), dtype=np.uint64)
    ctx = np.arange(C, dtype=np.uint32)[:, None].repeat(per, axis=1)
    rec = np.zeros((C, per), RECORD_DTYPE)
    rec["ts"], rec["ctx_key"], rec["region_id"], rec["kind"] = ts, ctx, region, kind
    # interleave the contexts `step` records at a time (trace buffers per warp)
    rec = rec.reshape(C, per // step, step).transpose(1, 0, 2).reshape(n)
    rec_u8 = rec.view(np.uint8).reshape(n, 16)
    p = dict(num_regions=6, num_classes=2, region_class=np.array([0, 1, 0, 1, 0xFF, 0], np.uint8),
             group_shift=4, num_groups=C >> 4)
    log(f"[gpu] staged run lists: n={n}, {256 // step} runs per chunk")
    g = gpu_run(rec_u8, p, with_plan=True)
    plan = g.pop("_plan")
    assert plan["runs"] == 1 and plan["unsorted"] == 0
    assert_parity(g, oracle_run(oracle_mod, rec_u8, p), what="staged run lists")


@pytest.mark.timeout(900)
def test_full_size_large_trace_whole(oracle_mod, tracegen_mod):
    """The 2^28-record trace (4 GiB, 1 % malformed markers, stack levels near
    10^3) run whole on the GPU and compared whole with the oracle: every
    counter, region statistic, overlap row, instance and exclusive time."""
    d = tracegen_mod.generate(5, threads=16)
    p = _params(d)
    rec = d["records"]
    n = len(rec)
    R = p["num_regions"]
    log(f"[gpu] full-size large trace: n={n}")
    g = gpu_run(rec, p)
    c = g["counters"].astype(np.uint64)
    assert int(c[31]) == 0, f"internal error flag {int(c[31])}"
    inst, excl = g["instances"], g["instance_excl"]
    log(f"[gpu] full-size large trace: max_level={int(c[14])}, mismatched={int(c[10])}; "
        "properties")
    # properties that hold at any size, checked first because they are cheap
    assert int(c[0]) == n and len(inst) == int(c[4])
    assert int(c[9]) + int(c[10]) + int(c[11]) == int(c[4])  # matched + mismatched + unclosed
    closed = inst["end_region_id"] != NO_END
    assert int(c[12]) + int(closed.sum()) == int(c[5])  # orphans + closed = ENDs
    assert np.all(excl[closed] <= (inst["t_end"][closed] - inst["t_begin"][closed]))
    rs = g["region_stats"].reshape(R, -1)
    ref = _region_stats_from_instances(inst, excl, R)
    for name, col in RS_FIELDS.items():
        if name != "orphan_end":
            np.testing.assert_array_equal(rs[:, col], ref[name], err_msg=f"region stats {name}")
    del ref
    log("[gpu] full-size large trace: oracle on the whole trace")
    o = oracle_run(oracle_mod, rec, p)
    log(f"[gpu] full-size large trace: oracle max_level={int(o['counters'][14])}; comparing")
    assert_parity(g, o, what="full cfg5")
