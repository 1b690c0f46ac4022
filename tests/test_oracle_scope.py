"""Pins of the oracle's iteration ordinals and scoped statistics
(oracle/argus_oracle_scope.cpp).

* hand-built traces with ordinals and scoped statistics derived by hand;
* a brute-force ordinal: for each instance, the earlier instances of the
  same context and BEGIN region are counted one by one, O(n^2);
* the scope that admits everything reproduces the unscoped per-region
  statistics of the (separately pinned) main oracle, orphan column aside;
* disjoint scopes partition the statistics: iteration windows [0, k) and
  [k, inf), or warp-role ranges, add up (sums and counts add, min and max
  combine) to the unscoped result.
"""
from __future__ import annotations

import numpy as np
import pytest

from golden_util import random_malformed, records_from_rows

B, E = 1, 2
RS_ORPHAN = 8


def _run(oracle_mod, rows, R):
    o = oracle_mod.run(records_from_rows(rows), R)
    return o, o["instances"], o["instance_excl"]


def test_hand_ordinals_and_window(oracle_mod):
    """ctx 0: regions 0, 1, 0, 2, 0 one after another (each 10 long); ctx 1:
    region 0 twice.  Ordinals 0 0 1 0 2 | 0 1.  The window of iterations
    [1, 1] keeps the second region-0 instance of each context: count 2,
    incl sum 20."""
    rows = []
    t = 0
    for r in (0, 1, 0, 2, 0):
        rows += [(t, 0, r, B), (t + 10, 0, r, E)]
        t += 20
    rows += [(0, 1, 0, B), (10, 1, 0, E), (20, 1, 0, B), (30, 1, 0, E)]
    _, inst, excl = _run(oracle_mod, rows, 3)
    s = oracle_mod.scope(inst, excl, 3)
    assert s["ordinal"].tolist() == [0, 0, 1, 0, 2, 0, 1]
    assert s["counters"].tolist()[:7] == [7, 7, 7, 0, 0, 0, 3]
    w = oracle_mod.scope(inst, excl, 3, iter_lo=1, iter_hi=1)
    assert w["stats"][0, :5].tolist() == [2, 20, 20, 10, 10]
    assert w["stats"][1, 0] == 0 and w["stats"][2, 0] == 0
    assert w["counters"].tolist()[:3] == [7, 2, 2]


def test_hand_role_group_and_region_mask(oracle_mod):
    """Four contexts (2 groups x 2 warps, group_shift 1), each one region-r
    instance of length 10 * (ctx + 1) with r = ctx % 2.  Warp role 1
    ((ctx & 1) == 1): contexts 1 and 3, region 1, incl 20 + 40.  Group 1:
    contexts 2 and 3.  Region mask {0}: contexts 0 and 2."""
    rows = []
    for c in range(4):
        rows += [(0, c, c % 2, B), (10 * (c + 1), c, c % 2, E)]
    _, inst, excl = _run(oracle_mod, rows, 2)
    role = oracle_mod.scope(inst, excl, 2, role_mask=1, role_lo=1, role_hi=1)
    assert role["stats"][1, :5].tolist() == [2, 60, 60, 20, 40] and role["stats"][0, 0] == 0
    grp = oracle_mod.scope(inst, excl, 2, group_shift=1, group_lo=1, group_hi=1)
    assert grp["stats"][0, :2].tolist() == [1, 30] and grp["stats"][1, :2].tolist() == [1, 40]
    msk = oracle_mod.scope(inst, excl, 2, region_mask=np.array([1, 0], np.uint8))
    assert msk["stats"][0, :2].tolist() == [2, 40] and msk["counters"][1] == 2


def test_hand_malformed_in_scope(oracle_mod):
    """A mismatched pair (BEGIN 0, END 1) and an unclosed BEGIN 1 in one
    context: in scope they are counted as mism_as_begin[0],
    mism_as_end[1] and unclosed[1]; no matched statistics."""
    _, inst, excl = _run(oracle_mod, [(0, 0, 0, B), (5, 0, 1, E), (6, 0, 1, B)], 2)
    s = oracle_mod.scope(inst, excl, 2)
    assert s["stats"][0, 9] == 1 and s["stats"][1, 10] == 1 and s["stats"][1, 7] == 1
    assert s["counters"].tolist()[:5] == [2, 2, 0, 1, 1]


def brute_ordinal(inst):
    out = []
    for x in range(len(inst)):
        out.append(sum(1 for y in range(x) if inst[y]["ctx_key"] == inst[x]["ctx_key"]
                       and inst[y]["region_id"] == inst[x]["region_id"]))
    return np.array(out, np.uint32)


@pytest.mark.parametrize("seed", range(30))
def test_brute_force_ordinal(oracle_mod, seed):
    rng = np.random.default_rng(700 + seed)
    R = 1 + seed % 4
    o = oracle_mod.run(random_malformed(rng, 120, 1 + seed % 3, R, [4, 30, 500][seed % 3]), R)
    s = oracle_mod.scope(o["instances"], o["instance_excl"], R)
    np.testing.assert_array_equal(s["ordinal"], brute_ordinal(o["instances"]))


def _combine(a, b):
    """Statistics of the union of two disjoint instance sets."""
    c = a + b
    for mn in (3, 5):
        c[:, mn] = np.minimum(a[:, mn], b[:, mn])
    for mx in (4, 6):
        c[:, mx] = np.maximum(a[:, mx], b[:, mx])
    return c


@pytest.mark.parametrize("seed", range(12))
def test_all_scope_and_partitions(oracle_mod, seed):
    rng = np.random.default_rng(800 + seed)
    R = 2 + seed % 5
    o = oracle_mod.run(random_malformed(rng, 600, 8, R, 2000), R)
    inst, excl = o["instances"], o["instance_excl"]
    full = oracle_mod.scope(inst, excl, R)
    want = o["region_stats"].copy()
    want[:, RS_ORPHAN] = 0
    np.testing.assert_array_equal(full["stats"], want)
    k = 1 + seed % 3
    lo = oracle_mod.scope(inst, excl, R, iter_hi=k - 1)
    hi = oracle_mod.scope(inst, excl, R, iter_lo=k)
    np.testing.assert_array_equal(_combine(lo["stats"], hi["stats"]), full["stats"])
    r0 = oracle_mod.scope(inst, excl, R, role_mask=7, role_lo=0, role_hi=2)
    r1 = oracle_mod.scope(inst, excl, R, role_mask=7, role_lo=3, role_hi=7)
    np.testing.assert_array_equal(_combine(r0["stats"], r1["stats"]), full["stats"])
    assert int(r0["counters"][1] + r1["counters"][1]) == len(inst)
