"""Pins of the oracle's PC-sample attribution (oracle/argus_oracle_samples.cpp).

What is pinned, and by what (none of it retypes the oracle's own code):
* hand-built traces whose owners, counts, alpha, m_hat and H are derived by
  hand below, with closed forms for H (Section 3.5: alpha = n / sum n,
  m_hat = sum alpha m, H = -sum alpha log alpha);
* a brute-force owner search, O(samples x instances): for each sample, every
  instance of its context is tested for "active at ts and matched", and the
  deepest one wins (Section 3.2: the innermost active region receives the
  execution count);
* closed forms: one owner gives H = 0 and alpha = 1; k owners with equal
  counts give H = ln k and alpha = 1/k;
* invariants: sum_r alpha = 1, sum_r m_hat = sum of m over the PCs that have
  an owner, weights are conserved (attributed + unattributed = total),
  H <= ln(owners).
"""
from __future__ import annotations

import math

import numpy as np
import pytest

from golden_util import random_malformed, records_from_rows

B, E = 1, 2


def _instances(oracle_mod, rows, R):
    return oracle_mod.run(records_from_rows(rows), R)["instances"]


def _samples(rows):
    s = np.zeros(len(rows), np.dtype([("ts", "<u8"), ("ctx_key", "<u4"), ("pc", "<u4")]))
    for i, (ts, ctx, pc) in enumerate(rows):
        s[i] = (ts, ctx, pc)
    return s


def test_hand_nested_shared_helper(oracle_mod):
    """ctx 0: region 0 over [0, 100) around region 1 over [20, 50).
    PC 7 (a shared helper) runs at 10 and 60 (under region 0) and at 30 and
    40 (under region 1): n = 2 / 2, alpha = 1/2 each, H = ln 2.
    PC 3 runs at 0 (region 0: begins are inclusive), 25 and 26 (region 1)
    and 100 (nothing: ends are exclusive): n = 1 / 2, alpha = 1/3 and 2/3,
    H = ln 3 - (2/3) ln 2; one unattributed execution.
    m(3) = 6, m(7) = 10: m_hat(0) = 10/2 + 6/3 = 7, m_hat(1) = 10/2 + 12/3 = 9."""
    inst = _instances(oracle_mod, [(0, 0, 0, B), (20, 0, 1, B), (50, 0, 1, E), (100, 0, 0, E)], 2)
    smp = _samples([(10, 0, 7), (30, 0, 7), (40, 0, 7), (60, 0, 7),
                    (0, 0, 3), (25, 0, 3), (26, 0, 3), (100, 0, 3)])
    m = np.zeros((1, 8))
    m[0, 3], m[0, 7] = 6.0, 10.0
    o = oracle_mod.samples(inst, smp, 2, 8, metrics=m)
    assert o["n"][7].tolist() == [2, 2] and o["n"][3].tolist() == [1, 2]
    assert o["pc_total"][7] == 4 and o["pc_total"][3] == 3
    assert o["pc_owners"].tolist() == [0, 0, 0, 2, 0, 0, 0, 2]
    assert o["alpha"][7].tolist() == [0.5, 0.5]
    assert o["alpha"][3].tolist() == [1 / 3, 2 / 3]
    assert o["entropy"][7] == pytest.approx(math.log(2), rel=1e-15)
    assert o["entropy"][3] == pytest.approx(math.log(3) - 2 / 3 * math.log(2), rel=1e-15)
    assert o["mhat"][0].tolist() == pytest.approx([7.0, 9.0], rel=1e-15)
    assert o["region_total"].tolist() == [3, 4]
    c = o["counters"]
    assert c.tolist()[:7] == [8, 0, 8, 7, 1, 0, 4]


def test_hand_mismatched_innermost(oracle_mod):
    """Region 0 over [0, 100) around a MISMATCHED pair [10, 50) (BEGIN region
    1, END region 2).  A sample at 20 has the mismatched instance innermost:
    it goes to region 0 and is counted as inner-unmatched.  A sample at 60
    goes to region 0 plainly."""
    inst = _instances(oracle_mod, [(0, 0, 0, B), (10, 0, 1, B), (50, 0, 2, E), (100, 0, 0, E)], 3)
    o = oracle_mod.samples(inst, _samples([(20, 0, 0), (60, 0, 0)]), 3, 1)
    assert o["n"][0].tolist() == [2, 0, 0]
    assert o["counters"].tolist()[:7] == [2, 0, 2, 2, 0, 1, 1]
    assert o["entropy"][0] == 0.0 and o["alpha"][0, 0] == 1.0


def test_hand_unclosed_and_zero_length(oracle_mod):
    """An UNCLOSED region 0 from 0 on, around region 1 over [10, 20) and a
    zero-length region 2 at [30, 30).  Samples at 15 -> region 1; at 5, 20,
    30 and 40 the only active instance is the unclosed one (a zero-length
    instance is never active): unattributed."""
    inst = _instances(oracle_mod, [(0, 0, 0, B), (10, 0, 1, B), (20, 0, 1, E),
                                   (30, 0, 2, B), (30, 0, 2, E)], 3)
    o = oracle_mod.samples(inst, _samples([(15, 0, 1), (5, 0, 1), (20, 0, 1), (30, 0, 1),
                                           (40, 0, 1)]), 3, 2)
    assert o["n"][1].tolist() == [0, 1, 0]
    assert o["counters"].tolist()[:7] == [5, 0, 5, 1, 4, 0, 1]


def test_hand_weights_contexts_and_bad_pcs(oracle_mod):
    """Two contexts with the same times: ctx 0 runs region 0 over [0, 10),
    ctx 1 runs region 1 over [0, 10).  PC 0 samples at 5 in ctx 0 (weight 3)
    and ctx 1 (weight 1): n = 3 / 1, alpha = 3/4 and 1/4,
    H = ln 4 - (3/4) ln 3.  A sample of ctx 2 (no instances) is unattributed;
    pc 9 >= P is bad and takes no part."""
    inst = _instances(oracle_mod, [(0, 0, 0, B), (10, 0, 0, E), (0, 1, 1, B), (10, 1, 1, E)], 2)
    smp = _samples([(5, 0, 0), (5, 1, 0), (5, 2, 0), (5, 0, 9)])
    w = np.array([3, 1, 2, 100], np.uint32)
    o = oracle_mod.samples(inst, smp, 2, 4, weights=w, metrics=np.array([[8.0, 0, 0, 0]]))
    assert o["n"][0].tolist() == [3, 1]
    assert o["alpha"][0].tolist() == [0.75, 0.25]
    assert o["entropy"][0] == pytest.approx(math.log(4) - 0.75 * math.log(3), rel=1e-15)
    assert o["mhat"][0].tolist() == [6.0, 2.0]
    assert o["counters"].tolist()[:7] == [4, 1, 6, 4, 2, 0, 2]


def brute_force(inst, smp, weights, R, P):
    """For each sample, test every instance of its context."""
    n = np.zeros((P, R), np.uint64)
    att = unatt = inner = bad = 0
    for i, s in enumerate(smp):
        w = int(weights[i]) if weights is not None else 1
        if int(s["pc"]) >= P:
            bad += 1
            continue
        ts = int(s["ts"])
        best, best_any = None, None
        for x in inst:
            if int(x["ctx_key"]) != int(s["ctx_key"]):
                continue
            closed = int(x["end_region_id"]) != 0xFFFF
            if not (int(x["t_begin"]) <= ts and (not closed or ts < int(x["t_end"]))):
                continue
            if best_any is None or int(x["level"]) > int(best_any["level"]):
                best_any = x
            if closed and int(x["end_region_id"]) == int(x["region_id"]):
                if best is None or int(x["level"]) > int(best["level"]):
                    best = x
        if best is None:
            unatt += w
            continue
        att += w
        if int(best_any["level"]) > int(best["level"]):
            inner += w
        n[int(s["pc"]), int(best["region_id"])] += np.uint64(w)
    return n, att, unatt, inner, bad


def random_samples(rng, n, n_ctx, ts_range, P):
    s = np.zeros(n, np.dtype([("ts", "<u8"), ("ctx_key", "<u4"), ("pc", "<u4")]))
    s["ts"] = rng.integers(0, ts_range, size=n)
    s["ctx_key"] = rng.integers(0, n_ctx + 1, size=n)
    s["pc"] = rng.integers(0, P + 1, size=n)  # pc == P is a bad PC
    return s


@pytest.mark.parametrize("seed", range(40))
def test_brute_force_owner(oracle_mod, seed):
    rng = np.random.default_rng(500 + seed)
    R, P, n_ctx, tr = 1 + seed % 5, 1 + seed % 7, 1 + seed % 3, [5, 20, 200][seed % 3]
    inst = oracle_mod.run(random_malformed(rng, 60, n_ctx, R, tr), R)["instances"]
    smp = random_samples(rng, 80, n_ctx, tr + 2, P)
    w = rng.integers(1, 5, size=len(smp)).astype(np.uint32) if seed % 2 else None
    o = oracle_mod.samples(inst, smp, R, P, weights=w)
    n, att, unatt, inner, bad = brute_force(inst, smp, w, R, P)
    np.testing.assert_array_equal(o["n"], n)
    c = o["counters"]
    assert (int(c[1]), int(c[3]), int(c[4]), int(c[5])) == (bad, att, unatt, inner)


def test_entropy_closed_forms(oracle_mod):
    """k regions side by side in k contexts, the same PC sampled equally
    often in each: alpha = 1/k and H = ln k; a PC with one owner has H = 0."""
    for k in (1, 2, 3, 5, 8):
        rows = []
        for r in range(k):
            rows += [(0, r, r, B), (10, r, r, E)]
        inst = _instances(oracle_mod, rows, k)
        smp = _samples([(t, r, 0) for r in range(k) for t in (1, 2, 3)] + [(4, 0, 1)])
        o = oracle_mod.samples(inst, smp, k, 2)
        assert o["entropy"][0] == pytest.approx(math.log(k), rel=1e-15, abs=0)
        assert o["alpha"][0].tolist() == pytest.approx([1 / k] * k, rel=1e-15)
        assert o["entropy"][1] == 0.0 and o["alpha"][1, 0] == 1.0


@pytest.mark.parametrize("seed", range(10))
def test_invariants(oracle_mod, seed):
    rng = np.random.default_rng(900 + seed)
    R, P = 6, 11
    inst = oracle_mod.run(random_malformed(rng, 400, 4, R, 300), R)["instances"]
    smp = random_samples(rng, 3000, 4, 320, P)
    w = rng.integers(1, 9, size=len(smp)).astype(np.uint32)
    m = rng.normal(size=(3, P))
    o = oracle_mod.samples(inst, smp, R, P, weights=w, metrics=m)
    c = o["counters"].astype(np.int64)
    assert c[2] == c[3] + c[4]  # weight conserved
    assert int(o["n"].sum()) == c[3] == int(o["pc_total"].sum()) == int(o["region_total"].sum())
    has = o["pc_total"] > 0
    np.testing.assert_allclose(o["alpha"][has].sum(axis=1), 1.0, rtol=1e-14)
    assert np.all(o["alpha"][~has] == 0)
    np.testing.assert_allclose(o["mhat"].sum(axis=1), m[:, has].sum(axis=1), rtol=1e-12, atol=1e-12)
    own = o["pc_owners"].astype(np.float64)
    assert np.all(o["entropy"] <= np.log(np.maximum(own, 1)) + 1e-12)
    assert np.all(o["entropy"] >= 0)
    assert int(c[6]) == int((o["n"] > 0).sum())


def test_mhat_strand_order(oracle_mod):
    """The sum over p is taken in 512 strands (p mod 512, each in increasing
    p) combined by halving.  One region owns PCs 0, 1 and 512 of P = 513,
    alpha = 1, metric 1e16, 1 and -1e16: strand 0 holds 1e16 + (-1e16) = 0,
    strand 1 holds 1, so m_hat = 1 exactly; adding in increasing p would lose
    the 1 to rounding (1e16 + 1 rounds to 1e16) and give 0.  A second metric,
    1e16, -1e16 and 1 on PCs 0, 256 and 1, checks the halving: its first step
    pairs strands 0 and 256 (0) before strand 1 joins (1), where pairing
    neighbours, or adding in increasing p, meets 1e16 + 1 first and gives 0."""
    inst = _instances(oracle_mod, [(0, 0, 0, B), (100, 0, 0, E)], 1)
    smp = _samples([(10, 0, 0), (10, 0, 1), (10, 0, 512), (10, 0, 256)])
    m = np.zeros((2, 513))
    m[0, 0], m[0, 1], m[0, 512] = 1e16, 1.0, -1e16
    m[1, 0], m[1, 256], m[1, 1] = 1e16, -1e16, 1.0
    o = oracle_mod.samples(inst, smp, 1, 513, metrics=m)
    assert o["alpha"][[0, 1, 256, 512], 0].tolist() == [1.0, 1.0, 1.0, 1.0]
    assert o["mhat"][0, 0] == 1.0
    assert o["mhat"][1, 0] == 1.0
