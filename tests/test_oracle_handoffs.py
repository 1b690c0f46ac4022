"""Pins of the oracle's phase-handoff gaps (oracle/argus_oracle_handoffs.cpp).

* hand-built traces: top-level phases and the phases inside two "step"
  regions, gaps and per-step totals derived by hand; phases of different
  parents are never paired; an unclosed phase is counted, not measured;
* brute force: for each level-L instance, its predecessor is searched among
  all earlier instances, O(n^2);
* time conservation on well-formed nested traces: a parent's inclusive time
  = lead-in before its first child + its children's inclusive times + the
  handoff gaps between them + the tail after its last child.
"""
from __future__ import annotations

import numpy as np
import pytest

from golden_util import random_malformed, random_wellformed, records_from_rows

B, E = 1, 2


def _inst(oracle_mod, rows, R):
    return oracle_mod.run(records_from_rows(rows), R)["instances"]


def test_hand_top_level(oracle_mod):
    """ctx 0: A [0, 10), B [15, 30), A [30, 50) at the top level, with a
    child C [16, 20) inside B; ctx 1: B [0, 7), A [100, 101).  Level 0 gaps:
    A->B 5, B->A 0 (ctx 0), B->A 93 (ctx 1).  Level 1: one phase only."""
    A, Bq, C = 0, 1, 2
    rows = [(0, 0, A, B), (10, 0, A, E), (15, 0, Bq, B), (16, 0, C, B), (20, 0, C, E),
            (30, 0, Bq, E), (30, 0, A, B), (50, 0, A, E), (0, 1, Bq, B), (7, 1, Bq, E),
            (100, 1, A, B), (101, 1, A, E)]
    inst = _inst(oracle_mod, rows, 3)
    h = oracle_mod.handoffs(inst, 3, 0)
    assert h["pairs"][A, Bq].tolist() == [1, 5, 5, 5]
    assert h["pairs"][Bq, A].tolist() == [2, 93, 0, 93]
    assert int(h["pairs"][:, :, 0].sum()) == 3
    assert h["counters"].tolist()[:3] == [5, 3, 98]
    assert h["hist"][0] == 1 and h["hist"][3] == 1 and h["hist"][7] == 1
    h1 = oracle_mod.handoffs(inst, 3, 1)
    assert h1["counters"].tolist()[:3] == [1, 0, 0]


def test_hand_steps(oracle_mod):
    """Two step regions S [0, 100) and [100, 200) with operator phases
    o1 [10, 20), o2 [25, 40), o3 [60, 70) and o1 [110, 120), o2 [121, 190).
    Level 1 gaps: 5, 20 in the first step (total 25), 1 in the second (1);
    the last phase of step 1 and the first of step 2 are not successive."""
    S, o1, o2, o3 = 0, 1, 2, 3
    rows = [(0, 0, S, B), (10, 0, o1, B), (20, 0, o1, E), (25, 0, o2, B), (40, 0, o2, E),
            (60, 0, o3, B), (70, 0, o3, E), (100, 0, S, E),
            (100, 0, S, B), (110, 0, o1, B), (120, 0, o1, E), (121, 0, o2, B), (190, 0, o2, E),
            (200, 0, S, E)]
    inst = _inst(oracle_mod, rows, 4)
    h = oracle_mod.handoffs(inst, 4, 1)
    assert h["parent_gap"].tolist() == [25, 0, 0, 0, 1, 0, 0]
    assert h["pairs"][o1, o2].tolist() == [2, 6, 1, 5]
    assert h["pairs"][o2, o3].tolist() == [1, 20, 20, 20]
    assert h["counters"].tolist()[:3] == [5, 3, 26]


def test_hand_malformed_phases(oracle_mod):
    """A mismatched top-level pair [0, 5) (BEGIN 0, END 1), then [8, 9) and
    a top-level BEGIN at 20 that never ends: gaps 3 (pair 0 -> 0) and 11
    (0 -> 1).  A BEGIN that never ends has no successor: the phases after it
    are nested inside it (one level deeper)."""
    rows = [(0, 0, 0, B), (5, 0, 1, E), (8, 0, 0, B), (9, 0, 0, E), (20, 0, 1, B)]
    h = oracle_mod.handoffs(_inst(oracle_mod, rows, 2), 2, 0)
    assert h["counters"].tolist()[:3] == [3, 2, 14]
    assert h["pairs"][0, 0].tolist() == [1, 3, 3, 3] and h["pairs"][0, 1].tolist() == [1, 11, 11, 11]
    rows2 = [(0, 0, 0, B), (5, 0, 1, B), (7, 0, 1, E), (8, 0, 1, B), (9, 0, 1, E)]
    inst2 = _inst(oracle_mod, rows2, 2)
    assert oracle_mod.handoffs(inst2, 2, 0)["counters"].tolist()[:3] == [1, 0, 0]
    h2 = oracle_mod.handoffs(inst2, 2, 1)
    assert h2["counters"].tolist()[:3] == [2, 1, 1] and h2["parent_gap"].tolist() == [1, 0, 0]


def brute(inst, R, L):
    pairs = {}
    for y in range(len(inst)):
        if int(inst[y]["level"]) != L:
            continue
        prev = None
        for x in range(y - 1, -1, -1):
            if int(inst[x]["level"]) == L and inst[x]["ctx_key"] == inst[y]["ctx_key"] and \
                    inst[x]["parent"] == inst[y]["parent"]:
                prev = x
                break
        if prev is None or int(inst[prev]["end_region_id"]) == 0xFFFF:
            continue
        k = (int(inst[prev]["region_id"]), int(inst[y]["region_id"]))
        pairs.setdefault(k, []).append((int(inst[y]["t_begin"]) - int(inst[prev]["t_end"])) % 2 ** 64)
    return pairs


@pytest.mark.parametrize("seed", range(24))
def test_brute_force(oracle_mod, seed):
    rng = np.random.default_rng(1700 + seed)
    R = 1 + seed % 4
    inst = oracle_mod.run(random_malformed(rng, 90, 1 + seed % 3, R, [10, 100, 1000][seed % 3]), R)["instances"]
    L = seed % 3
    h = oracle_mod.handoffs(inst, R, L)
    want = brute(inst, R, L)
    for a in range(R):
        for b in range(R):
            v = want.get((a, b), [])
            got = h["pairs"][a, b].tolist()
            exp = [len(v), sum(v) % 2 ** 64, min(v) if v else 2 ** 64 - 1, max(v) if v else 0]
            assert got == exp, (a, b, got, exp)


@pytest.mark.parametrize("seed", range(10))
def test_time_conservation(oracle_mod, seed):
    rng = np.random.default_rng(1800 + seed)
    R = 3
    rec, _ = random_wellformed(rng, 3, 40, R, max_depth=4, t_spread=9)
    o = oracle_mod.run(rec, R)
    inst = o["instances"]
    for L in (1, 2, 3):
        h = oracle_mod.handoffs(inst, R, L)
        kids = {}
        for y in range(len(inst)):
            if int(inst[y]["level"]) == L:
                kids.setdefault(int(inst[y]["parent"]), []).append(y)
        for p, ch in kids.items():
            first, last = inst[ch[0]], inst[ch[-1]]
            incl = sum(int(inst[c]["t_end"]) - int(inst[c]["t_begin"]) for c in ch)
            lead = int(first["t_begin"]) - int(inst[p]["t_begin"])
            tail = int(inst[p]["t_end"]) - int(last["t_end"])
            assert lead + incl + int(h["parent_gap"][p]) + tail == \
                int(inst[p]["t_end"]) - int(inst[p]["t_begin"])
