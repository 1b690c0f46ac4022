"""Pins for the CPU oracle: it is checked against things other than itself.

* hand-derived results of the hand-built traces in tests/golden/ (each case
  carries its derivation and the passage it follows);
* an independent derivation of the matcher (clamped depth scan and
  (level, ctx) adjacency, instead of an explicit stack);
* an independent derivation of exclusive time (time attributed to the
  innermost open instance between consecutive markers, Section 3.2);
* O(n^2) brute-force overlap from known intervals, and the K = 1 special
  case that reduces to the textbook length of a union of intervals;
* the generator's own instance lists for the well-formed configurations;
* invariants I1-I12 (matched instances equal matched begins, exclusive <=
  inclusive, unmatched markers reported, ...) on random malformed traces.
"""
from __future__ import annotations

import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

from golden_util import (INSTANCE_DTYPE, NONE32, RS_FIELDS, RS_HIST_EXCL, RS_HIST_INCL,
                         U64_MAX, case_params, expected_counters, expected_instances,
                         expected_region_stats, load_cases, random_malformed,
                         random_wellformed, records_from_rows)

CASES = load_cases()


def run_oracle(oracle_mod, rec, **p):
    return oracle_mod.run(rec, p["num_regions"], p.get("num_classes", 0),
                          p.get("region_class"), p.get("group_shift", 0),
                          p.get("num_groups", 0))


# ------------------------------------------------------------- hand-built traces

@pytest.mark.parametrize("case", CASES, ids=[c["name"] for c in CASES])
def test_hand_trace(oracle_mod, case):
    rec = records_from_rows(case["records"])
    p = case_params(case)
    out = run_oracle(oracle_mod, rec, **p)
    np.testing.assert_array_equal(out["counters"], expected_counters(case))
    if "region_stats" in case:
        np.testing.assert_array_equal(out["region_stats"], expected_region_stats(case))
    if "instances" in case:
        exp = expected_instances(case)
        assert out["instances"].tobytes() == exp.tobytes()
        np.testing.assert_array_equal(out["instance_excl"], np.array(case["excl"], np.uint64))
    if "overlap_group" in case:
        np.testing.assert_array_equal(out["overlap_group"],
                                      np.array(case["overlap_group"], np.uint64))
        np.testing.assert_array_equal(out["overlap_global"],
                                      np.array(case["overlap_global"], np.uint64))


# ------------------------------------------------ independent matcher derivation

def scan_derivation(rec_u8: np.ndarray, R: int):
    """Instances and exclusive times by a different route than a stack.

    Per context (records in (ctx, ts, input index) order) the clamped depth
    s_i = max(0, s_{i-1} + delta_i) is the stack size after record i; an END
    with s_{i-1} = 0 is an orphan.  A BEGIN's level is s_{i-1}, a non-orphan
    END's level is s_i.  Within one (ctx, level) group, kinds alternate B, E,
    B, E, ..., so a BEGIN pairs with the next record of its group when that
    is an END.  The parent of a BEGIN at level L is the last BEGIN at level
    L-1 before it.  Exclusive time: every gap between consecutive records of
    a context belongs to the innermost open instance after the first of the
    two records.
    """
    r = rec_u8.reshape(-1).view(np.dtype([("ts", "<u8"), ("ctx", "<u4"), ("reg", "<u2"),
                                          ("kind", "u1"), ("pad", "u1")]))
    seq = np.arange(len(r))
    valid = ((r["kind"] == 1) | (r["kind"] == 2)) & (r["reg"] < R)
    idx = seq[valid]
    order = idx[np.lexsort((idx, r["ts"][idx], r["ctx"][idx]))]
    ts = r["ts"][order].astype(object)
    ctx = r["ctx"][order]
    reg = r["reg"][order]
    isb = r["kind"][order] == 1
    n = len(order)
    begin_rank = np.cumsum(isb) - isb  # exclusive count of BEGINs
    inst = []
    excl_by_id = {}
    start = 0
    while start < n:
        end = start
        while end < n and ctx[end] == ctx[start]:
            end += 1
        s_prev = 0
        level = {}
        orphan = set()
        s_after = {}
        for i in range(start, end):
            if isb[i]:
                level[i] = s_prev
                s_prev += 1
            elif s_prev == 0:
                orphan.add(i)
            else:
                s_prev -= 1
                level[i] = s_prev
            s_after[i] = s_prev
        # group by level, in position order
        groups = {}
        for i in range(start, end):
            if i in orphan:
                continue
            groups.setdefault(level[i], []).append(i)
        partner = {}
        for L, members in groups.items():
            for a, b in zip(members, members[1:]):
                if isb[a] and not isb[b]:
                    partner[a] = b
        last_begin_at = {}
        parent_pos = {}
        owner_after = {}
        for i in range(start, end):
            if isb[i]:
                L = level[i]
                parent_pos[i] = last_begin_at.get(L - 1) if L > 0 else None
                last_begin_at[L] = i
            # innermost open BEGIN after record i is the last BEGIN at level s_after-1
            sa = s_after[i]
            owner_after[i] = last_begin_at.get(sa - 1) if sa > 0 else None
        gap_sum = {}
        for i in range(start, end - 1):
            o = owner_after[i]
            if o is not None:
                gap_sum[o] = gap_sum.get(o, 0) + (ts[i + 1] - ts[i])
        for i in range(start, end):
            if not isb[i]:
                continue
            pid = parent_pos[i]
            parent = int(begin_rank[pid]) if pid is not None else NONE32
            if i in partner:
                j = partner[i]
                t_end, ereg = ts[j], int(reg[j])
                excl = gap_sum.get(i, 0)
            else:
                t_end, ereg = U64_MAX, 0xFFFF
                excl = 0
            inst.append((int(ts[i]), int(t_end), int(ctx[i]), parent, level[i], int(reg[i]), ereg))
            excl_by_id[len(inst) - 1] = excl
        start = end
    a = np.zeros(len(inst), INSTANCE_DTYPE)
    for i, row in enumerate(inst):
        a[i] = row
    return a, np.array([excl_by_id[i] for i in range(len(inst))], np.uint64)


@settings(max_examples=300, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(seed=st.integers(0, 2**32 - 1), n=st.integers(0, 64), n_ctx=st.integers(1, 4),
       R=st.integers(1, 5), ts_range=st.sampled_from([3, 10, 1000]))
def test_matcher_matches_depth_scan_derivation(oracle_mod, seed, n, n_ctx, R, ts_range):
    rng = np.random.default_rng(seed)
    rec = random_malformed(rng, n, n_ctx, R, ts_range)
    out = run_oracle(oracle_mod, rec, num_regions=R)
    inst, excl = scan_derivation(rec, R)
    assert out["instances"].tobytes() == inst.tobytes()
    np.testing.assert_array_equal(out["instance_excl"], excl)


def test_flat_trace_pairs_consecutive_records(oracle_mod):
    """Depth-1 special case: alternating B/E per context pair up in order."""
    rng = np.random.default_rng(7)
    rows, ivs = [], []
    for ctx in range(5):
        t = 0
        for k in range(40):
            reg = int(rng.integers(0, 3))
            t0 = t + int(rng.integers(1, 9))
            t1 = t0 + int(rng.integers(1, 9))  # positive: the input is shuffled
            rows += [(t0, ctx, reg, 1), (t1, ctx, reg, 2)]
            ivs.append((t0, t1, ctx, NONE32, 0, reg, reg))
            t = t1
    perm = rng.permutation(len(rows))
    rec = records_from_rows([rows[i] for i in perm])
    out = run_oracle(oracle_mod, rec, num_regions=3)
    exp = np.array(ivs, INSTANCE_DTYPE)
    assert out["instances"].tobytes() == exp.tobytes()
    np.testing.assert_array_equal(out["instance_excl"], (exp["t_end"] - exp["t_begin"]))


# ------------------------------------------------------- brute-force overlap

def brute_force_overlap(ivs, K, cls, group_shift, G):
    """O(n^2) overlap from a list of (ctx, region, t0, t1) intervals."""
    U = np.zeros((G, K, K), object)
    Q = np.zeros((G, K, K), object)
    for g in range(G):
        mine = [(cls[reg], t0, t1) for (ctx, reg, t0, t1, *_) in ivs
                if (ctx >> group_shift) == g and cls[reg] < K]
        # Q: pairwise intersections
        for i in range(len(mine)):
            for j in range(len(mine)):
                if i == j:
                    continue
                a, b = mine[i], mine[j]
                inter = max(0, min(a[2], b[2]) - max(a[1], b[1]))
                if a[0] == b[0]:
                    if i < j:
                        Q[g, a[0], a[0]] += inter
                else:
                    Q[g, a[0], b[0]] += inter
        # U: elementary intervals
        pts = sorted({p for (_, t0, t1) in mine for p in (t0, t1)})
        for lo, hi in zip(pts, pts[1:]):
            act = [any(c == k and t0 <= lo and hi <= t1 for (c, t0, t1) in mine) for k in range(K)]
            for A in range(K):
                for B in range(K):
                    if act[A] and act[B]:
                        U[g, A, B] += hi - lo
    return U, Q


@settings(max_examples=150, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(seed=st.integers(0, 2**32 - 1), n_ctx=st.integers(1, 6), pairs=st.integers(0, 8),
       K=st.integers(1, 3), shift=st.integers(0, 2), G=st.integers(1, 3),
       depth=st.integers(1, 3))
def test_overlap_brute_force(oracle_mod, seed, n_ctx, pairs, K, shift, G, depth):
    rng = np.random.default_rng(seed)
    R = 4
    cls = rng.integers(0, K + 1, size=R).astype(np.uint8)  # value K = unclassified
    rec, ivs = random_wellformed(rng, n_ctx, pairs, R, max_depth=depth, t_spread=20)
    out = run_oracle(oracle_mod, rec, num_regions=R, num_classes=K, region_class=cls,
                     group_shift=shift, num_groups=G)
    U, Q = brute_force_overlap(ivs, K, cls, shift, G)
    og = out["overlap_group"]
    np.testing.assert_array_equal(og[:, 0].astype(object), U)
    np.testing.assert_array_equal(og[:, 1].astype(object), Q)
    np.testing.assert_array_equal(out["overlap_global"][0].astype(object), U.sum(axis=0))
    np.testing.assert_array_equal(out["overlap_global"][1].astype(object), Q.sum(axis=0))
    skipped = sum(1 for (ctx, reg, *_r) in ivs if cls[reg] < K and (ctx >> shift) >= G)
    assert int(out["counters"][15]) == skipped


def test_single_class_union_length(oracle_mod):
    """K = 1: U[0][0] of a group is the length of the union of its intervals."""
    rng = np.random.default_rng(11)
    rec, ivs = random_wellformed(rng, 8, 30, 3, max_depth=3, t_spread=40)
    cls = np.zeros(3, np.uint8)
    out = run_oracle(oracle_mod, rec, num_regions=3, num_classes=1, region_class=cls,
                     group_shift=3, num_groups=1)
    spans = sorted((t0, t1) for (_, _, t0, t1, _) in ivs if t1 > t0)
    total, cur_lo, cur_hi = 0, None, None
    for lo, hi in spans:
        if cur_hi is None or lo > cur_hi:
            if cur_hi is not None:
                total += cur_hi - cur_lo
            cur_lo, cur_hi = lo, hi
        else:
            cur_hi = max(cur_hi, hi)
    if cur_hi is not None:
        total += cur_hi - cur_lo
    assert int(out["overlap_group"][0, 0, 0, 0]) == total


# ------------------------------------------------------------------ invariants

def check_invariants(out, R, wellformed=False, depth_bound=None):
    c = {n: int(out["counters"][i]) for i, n in enumerate(
        ["n_records", "n_valid", "n_bad_kind", "n_bad_region", "n_begin", "n_end", "ts_min",
         "ts_max", "n_ctx", "n_matched", "n_mismatched", "n_unclosed", "n_orphan_end",
         "n_self_nested", "max_level", "n_overlap_skipped"])}
    rs = out["region_stats"].astype(object)
    inst, excl = out["instances"], out["instance_excl"]
    # I1
    assert c["n_records"] == c["n_valid"] + c["n_bad_kind"] + c["n_bad_region"]
    assert c["n_valid"] == c["n_begin"] + c["n_end"]
    # I2, I3
    assert c["n_begin"] == c["n_matched"] + c["n_mismatched"] + c["n_unclosed"]
    assert c["n_end"] == c["n_matched"] + c["n_mismatched"] + c["n_orphan_end"]
    assert len(inst) == c["n_begin"]
    # I4
    assert sum(rs[:, RS_FIELDS["count"]]) == c["n_matched"]
    assert rs[:, RS_HIST_INCL:RS_HIST_INCL + 65].sum() == c["n_matched"]
    assert rs[:, RS_HIST_EXCL:RS_HIST_EXCL + 65].sum() == c["n_matched"]
    # I5: exclusive <= inclusive, children's sum <= parent
    closed = inst["end_region_id"] != 0xFFFF
    incl = (inst["t_end"] - inst["t_begin"])
    assert np.all(excl[closed] <= incl[closed])
    assert np.all(excl[~closed] == 0)
    # I6
    for r in range(R):
        if rs[r, RS_FIELDS["count"]] > 0:
            assert rs[r, RS_FIELDS["incl_min"]] <= rs[r, RS_FIELDS["incl_max"]]
            assert rs[r, RS_FIELDS["excl_min"]] <= rs[r, RS_FIELDS["excl_max"]]
            assert rs[r, RS_FIELDS["excl_sum"]] <= rs[r, RS_FIELDS["incl_sum"]]
        else:
            assert rs[r, RS_FIELDS["incl_min"]] == U64_MAX and rs[r, RS_FIELDS["incl_max"]] == 0
    # I7
    assert sum(rs[:, RS_FIELDS["unclosed"]]) == c["n_unclosed"]
    assert sum(rs[:, RS_FIELDS["orphan_end"]]) == c["n_orphan_end"]
    assert sum(rs[:, RS_FIELDS["mism_as_begin"]]) == c["n_mismatched"]
    assert sum(rs[:, RS_FIELDS["mism_as_end"]]) == c["n_mismatched"]
    assert sum(rs[:, RS_FIELDS["self_nested"]]) == c["n_self_nested"]
    if wellformed:
        # I8
        assert c["n_mismatched"] == c["n_unclosed"] == c["n_orphan_end"] == 0
        assert c["n_matched"] * 2 == c["n_valid"]
        # I9: per context, sum of exclusive = sum of inclusive of level-0 instances
        for ctx in np.unique(inst["ctx_key"]):
            m = inst["ctx_key"] == ctx
            top = m & (inst["level"] == 0)
            assert int(excl[m].astype(object).sum()) == int(incl[top].astype(object).sum())
        # I12
        if depth_bound is not None:
            assert c["max_level"] < depth_bound
    if "overlap_group" in out:
        og = out["overlap_group"].astype(object)
        K = og.shape[-1]
        for g in range(og.shape[0]):
            U, Q = og[g, 0], og[g, 1]
            for A in range(K):
                for B in range(K):
                    # I10
                    assert U[A, B] == U[B, A] and Q[A, B] == Q[B, A]
                    assert U[A, B] <= min(U[A, A], U[B, B])
                    if A != B:
                        assert Q[A, B] >= U[A, B]
        np.testing.assert_array_equal(out["overlap_global"].astype(object), og.sum(axis=0))


@settings(max_examples=300, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(seed=st.integers(0, 2**32 - 1), n=st.integers(0, 64), n_ctx=st.integers(1, 4),
       R=st.integers(1, 5), ts_range=st.sampled_from([3, 10, 1000]), K=st.integers(0, 3))
def test_invariants_random_malformed(oracle_mod, seed, n, n_ctx, R, ts_range, K):
    rng = np.random.default_rng(seed)
    rec = random_malformed(rng, n, n_ctx, R, ts_range)
    cls = rng.integers(0, K + 1, size=R).astype(np.uint8)
    out = run_oracle(oracle_mod, rec, num_regions=R, num_classes=K, region_class=cls,
                     group_shift=1, num_groups=2)
    check_invariants(out, R)


@settings(max_examples=100, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(seed=st.integers(0, 2**32 - 1), n_ctx=st.integers(1, 5), pairs=st.integers(0, 20),
       depth=st.integers(1, 5))
def test_invariants_wellformed_and_permutation(oracle_mod, seed, n_ctx, pairs, depth):
    rng = np.random.default_rng(seed)
    R = 4
    rec, ivs = random_wellformed(rng, n_ctx, pairs, R, max_depth=depth)
    cls = np.array([0, 1, 0, 2], np.uint8)
    out = run_oracle(oracle_mod, rec, num_regions=R, num_classes=2, region_class=cls,
                     group_shift=1, num_groups=4)
    check_invariants(out, R, wellformed=True, depth_bound=depth)
    # I11: (ctx, ts) keys are distinct here, so any input order gives the same outputs
    rec2 = rec[rng.permutation(len(rec))]
    out2 = run_oracle(oracle_mod, rec2, num_regions=R, num_classes=2, region_class=cls,
                      group_shift=1, num_groups=4)
    for k in out:
        np.testing.assert_array_equal(out[k], out2[k])
    # the intervals the trace was built from are exactly the matched instances
    exp = sorted((ctx, t0, t1, reg, lvl) for (ctx, reg, t0, t1, lvl) in ivs)
    got = sorted(zip(out["instances"]["ctx_key"].tolist(), out["instances"]["t_begin"].tolist(),
                     out["instances"]["t_end"].tolist(), out["instances"]["region_id"].tolist(),
                     out["instances"]["level"].tolist()))
    assert got == exp


# ------------------------------------------------------------ generator truth

@pytest.mark.parametrize("cfg,kw", [(1, {}), (2, dict(blocks=3)), (4, dict(blocks=3))])
def test_generator_ground_truth(oracle_mod, tracegen_mod, cfg, kw):
    d = tracegen_mod.generate(cfg, truth=True, **kw)
    out = oracle_mod.run(d["records"], d["num_regions"], d["num_classes"], d["region_class"],
                         d["group_shift"], d["num_groups"])
    truth = d["truth"]
    assert out["instances"].tobytes() == truth.tobytes()
    R = d["num_regions"]
    check_invariants(out, R, wellformed=True, depth_bound={1: 3, 2: 2, 4: 1}[cfg])
    # statistics are direct sums over the generator's own instance list
    incl = (truth["t_end"] - truth["t_begin"]).astype(np.uint64)
    child = np.zeros(len(truth), np.uint64)
    has_p = truth["parent"] != NONE32
    np.add.at(child, truth["parent"][has_p], incl[has_p])
    excl = incl - child
    np.testing.assert_array_equal(out["instance_excl"], excl)
    rs = out["region_stats"]
    for r in range(R):
        m = truth["region_id"] == r
        assert int(rs[r, RS_FIELDS["count"]]) == int(m.sum())
        assert int(rs[r, RS_FIELDS["incl_sum"]]) == int(incl[m].astype(object).sum())
        assert int(rs[r, RS_FIELDS["excl_sum"]]) == int(excl[m].astype(object).sum())
        if m.any():
            assert int(rs[r, RS_FIELDS["incl_min"]]) == int(incl[m].min())
            assert int(rs[r, RS_FIELDS["excl_max"]]) == int(excl[m].max())
        bins_i = np.array([int(v).bit_length() for v in incl[m]], int)
        bins_e = np.array([int(v).bit_length() for v in excl[m]], int)
        np.testing.assert_array_equal(rs[r, RS_HIST_INCL:RS_HIST_INCL + 65],
                                      np.bincount(bins_i, minlength=65))
        np.testing.assert_array_equal(rs[r, RS_HIST_EXCL:RS_HIST_EXCL + 65],
                                      np.bincount(bins_e, minlength=65))


def test_generator_malformed_shapes(oracle_mod, tracegen_mod):
    """Configs 3 and 5 carry injected faults: invariants hold and ambiguity > 0."""
    for cfg, kw in [(3, dict(blocks=2)), (5, dict(blocks=16, size=1 << 18))]:
        d = tracegen_mod.generate(cfg, **kw)
        out = oracle_mod.run(d["records"], d["num_regions"], d["num_classes"],
                             d["region_class"], d["group_shift"], d["num_groups"])
        check_invariants(out, d["num_regions"])
        c = out["counters"]
        assert int(c[10]) + int(c[11]) > 0  # mismatched + unclosed
        if cfg == 3:
            assert int(c[13]) > 0  # self-nested: later tokens nest inside a stuck token
