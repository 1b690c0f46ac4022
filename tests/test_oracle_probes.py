"""Pins of the oracle's probe <-> reference join (oracle/argus_oracle_probes.cpp).

* hand-built references and probes: latencies 10..50 give, by hand,
  p0 = 10, p20 = 10, p40 = 20, p60 = 30, p80 = 40, p100 = 50, mean 30;
  joins go by (context, operation, iteration) even when the probe run's
  clock is far from the reference's; bad and unjoined probes are counted;
* brute force: the iteration is found by counting earlier instances, and
  each percentile as the smallest latency x with #{latency <= x} >= k, by
  counting, O(n^2) -- no sort involved;
* invariants: joined + unjoined + bad = probes; group counts add up to the
  joined probes; p0 <= p20 <= ... <= p100; min <= mean <= max.
"""
from __future__ import annotations

import numpy as np
import pytest

from golden_util import random_malformed, records_from_rows

B, E = 1, 2


def _probes(rows):
    import oracle
    a = np.zeros(len(rows), oracle.PROBE_DTYPE)
    for i, (ts, te, ctx, it, op) in enumerate(rows):
        a[i]["t_start"], a[i]["t_end"], a[i]["ctx_key"] = ts, te, ctx
        a[i]["iteration"], a[i]["op_region"] = it, op
    return a


def _ref(oracle_mod):
    """ctx 0: region 1 (a TMA load) issued at 100, 200, 300 (iterations 0,
    1, 2), each inside a region-0 mainloop instance; ctx 1: region 1 once at
    1000."""
    rows = []
    for i, t in enumerate((100, 200, 300)):
        rows += [(t - 5, 0, 0, B), (t, 0, 1, B), (t + 50, 0, 1, E), (t + 60, 0, 0, E)]
    rows += [(1000, 1, 1, B), (1010, 1, 1, E)]
    return oracle_mod.run(records_from_rows(rows), 2)["instances"]


def test_hand_percentiles_and_join(oracle_mod):
    inst = _ref(oracle_mod)
    # instance indices: ctx 0 -> 0 (r0), 1 (r1 it0), 2 (r0), 3 (r1 it1), 4 (r0), 5 (r1 it2); ctx 1 -> 6
    lat = [30, 10, 50, 20, 40]
    rows = [(10 ** 9 + k, 10 ** 9 + k + d, 0, 1, 1) for k, d in enumerate(lat)]  # iteration 1
    rows += [(5, 12, 1, 0, 1)]          # ctx 1, iteration 0 -> instance 6, latency 7
    rows += [(0, 3, 0, 3, 1)]           # iteration 3 does not exist: unjoined
    rows += [(0, 3, 2, 0, 1)]           # context 2 has no instances: unjoined
    rows += [(9, 3, 0, 0, 1)]           # t_end < t_start: bad
    rows += [(0, 3, 0, 0, 7)]           # region 7 >= R: bad
    o = oracle_mod.probes(inst, 2, _probes(rows))
    assert o["ref"].tolist() == [3, 3, 3, 3, 3, 6, 2 ** 32 - 1, 2 ** 32 - 1, 2 ** 32 - 1, 2 ** 32 - 1]
    assert o["completion"][:6].tolist() == [230, 210, 250, 220, 240, 1007]
    assert o["counters"].tolist()[:5] == [10, 2, 6, 2, 2]
    assert o["groups"].tolist() == [[3, 5, 150, 200, 10, 10, 20, 30, 40, 50],
                                    [6, 1, 7, 1000, 7, 7, 7, 7, 7, 7]]
    assert o["mean"].tolist() == [30.0, 7.0]


def test_hand_small_counts(oracle_mod):
    """Nearest rank with n = 2 (latencies 4, 9): ranks 1, 1, 1, 2, 2, 2;
    with n = 3 (1, 2, 3): ranks 1, 1, 2, 2, 3, 3."""
    inst = _ref(oracle_mod)
    o = oracle_mod.probes(inst, 2, _probes([(0, 9, 0, 0, 1), (0, 4, 0, 0, 1),
                                            (0, 3, 0, 2, 1), (0, 1, 0, 2, 1), (0, 2, 0, 2, 1)]))
    assert o["groups"][:, 4:].tolist() == [[4, 4, 4, 9, 9, 9], [1, 1, 2, 2, 3, 3]]
    assert o["mean"].tolist() == [6.5, 2.0]


def brute(inst, R, pr):
    """Join by counting earlier instances; percentiles by counting."""
    groups = {}
    ref = []
    for p in pr:
        if int(p["t_end"]) < int(p["t_start"]) or int(p["op_region"]) >= R:
            ref.append(None)
            continue
        hit = None
        seen = 0
        for x in range(len(inst)):
            if int(inst[x]["ctx_key"]) == int(p["ctx_key"]) and \
                    int(inst[x]["region_id"]) == int(p["op_region"]):
                if seen == int(p["iteration"]):
                    hit = x
                    break
                seen += 1
        ref.append(hit)
        if hit is not None:
            groups.setdefault(hit, []).append(int(p["t_end"]) - int(p["t_start"]))
    rows = []
    for x in sorted(groups):
        v = groups[x]
        n = len(v)
        row = [x, n, sum(v) % 2 ** 64, int(inst[x]["t_begin"])]
        for q in (0, 20, 40, 60, 80, 100):
            k = max(1, -(-q * n // 100))
            row.append(min(c for c in v if sum(1 for d in v if d <= c) >= k))
        rows.append(row)
    return ref, rows


@pytest.mark.parametrize("seed", range(25))
def test_brute_force(oracle_mod, seed):
    import oracle
    rng = np.random.default_rng(1300 + seed)
    R, n_ctx = 1 + seed % 4, 1 + seed % 3
    inst = oracle_mod.run(random_malformed(rng, 80, n_ctx, R, [10, 100, 1000][seed % 3]), R)["instances"]
    m = 60
    pr = np.zeros(m, oracle.PROBE_DTYPE)
    pr["t_start"] = rng.integers(0, 50, size=m)
    pr["t_end"] = pr["t_start"] + rng.integers(-3, 12, size=m)
    pr["ctx_key"] = rng.integers(0, n_ctx + 1, size=m)
    pr["iteration"] = rng.integers(0, 6, size=m)
    pr["op_region"] = rng.integers(0, R + 1, size=m)
    o = oracle_mod.probes(inst, R, pr)
    ref, rows = brute(inst, R, pr)
    assert o["ref"].tolist() == [2 ** 32 - 1 if r is None else r for r in ref]
    assert o["groups"].tolist() == rows
    c = o["counters"]
    assert int(c[1] + c[2] + c[3]) == m and int(o["groups"][:, 1].sum()) == int(c[2])
    g = o["groups"]
    if len(g):
        assert np.all(g[:, 5:10] >= g[:, 4:9])
        assert np.all((o["mean"] >= g[:, 4]) & (o["mean"] <= g[:, 9]))
