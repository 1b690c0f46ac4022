"""The pins must catch plausible mistakes in the oracle.

Each mutant is a one-line textual change to a COPY of one oracle source
(a dropped term, a wrong sign, index or comparison), compiled with the other
source into a temporary library.  The pin checks (hand-built traces, the
depth-scan derivation, the brute-force overlap and owner searches, closed
forms and invariants) are run against it and at least one of them must fail.
The real oracle is never modified.
"""
from __future__ import annotations

import os
import subprocess

import numpy as np
import pytest

from golden_util import (case_params, expected_counters, expected_instances,
                         expected_region_stats, load_cases, random_malformed,
                         random_wellformed, records_from_rows)
from test_oracle_pins import brute_force_overlap, check_invariants, scan_derivation

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "argus_oracle.cpp")
SRC_S = os.path.join(ROOT, "oracle", "argus_oracle_samples.cpp")
SRC_C = os.path.join(ROOT, "oracle", "argus_oracle_scope.cpp")
SRC_P = os.path.join(ROOT, "oracle", "argus_oracle_probes.cpp")
SRC_H = os.path.join(ROOT, "oracle", "argus_oracle_handoffs.cpp")
SOURCES = (SRC, SRC_S, SRC_C, SRC_P, SRC_H)

# one-line mutants of the phase handoffs (argus_oracle_handoffs.cpp)
MUTANTS_H = {
    "parent_ignored": ("const std::pair<uint32_t, uint32_t> key{b.ctx, b.parent};",
                       "const std::pair<uint32_t, uint32_t> key{b.ctx, 0u};"),
    "gap_from_begin": ("const uint64_t gap = b.t_begin - a.t_end;",
                       "const uint64_t gap = b.t_begin - a.t_begin;"),
    "level_off_by_one": ("if (b.level != level) continue;", "if (b.level != level + 1) continue;"),
    "gap_to_child": ("parent_gap[b.parent] += gap;", "parent_gap[y] += gap;"),
    "min_sentinel_zero": ("pairs[4 * i + 2] = ~uint64_t(0);", "pairs[4 * i + 2] = 0;"),
    "first_child_kept": ("    last[key] = y;\n", "    if (it == last.end()) last[key] = y;\n"),
    "pair_transposed": ("pairs + 4 * (uint64_t(a.region) * R + b.region)",
                        "pairs + 4 * (uint64_t(b.region) * R + a.region)"),
}

# one-line mutants of the probe join (argus_oracle_probes.cpp)
MUTANTS_P = {
    "join_first_iteration": ("const uint32_t x = it->second[p.iteration];",
                             "const uint32_t x = it->second[0];"),
    "rank_floor": ("uint64_t rank = (uint64_t(q[k]) * n + 99) / 100;",
                   "uint64_t rank = (uint64_t(q[k]) * n) / 100;"),
    "end_before_start_accepted": ("if (p.t_end < p.t_start || p.op_region >= num_regions) {",
                                  "if (p.op_region >= num_regions) {"),
    "completion_from_end": ("completion[j] = inst[x].t_begin + lat;",
                            "completion[j] = inst[x].t_end + lat;"),
    "mean_truncated": ("mean[g] = double(sum) / double(n);", "mean[g] = double(sum / n);"),
    "latencies_unsorted": ("std::sort(v.begin(), v.end());", "(void)0;"),
    "join_ignores_context": ("auto it = by_key.find({p.ctx, p.op_region});",
                             "auto it = by_key.find({0u, p.op_region});"),
    "iteration_off_by_one": ("p.iteration >= it->second.size()",
                             "p.iteration + 1 >= it->second.size()"),
}

# one-line mutants of the scopes and ordinals (argus_oracle_scope.cpp)
MUTANTS_C = {
    "ordinal_off_by_one": ("    ordinal[x] = c;\n", "    ordinal[x] = c + 1;\n"),
    "ordinal_per_context_only": ("seen[{inst[x].ctx, inst[x].region}]", "seen[{inst[x].ctx, 0}]"),
    "window_exclusive": ("in_range(ordinal[x], sc->iter_lo, sc->iter_hi)",
                         "in_range(ordinal[x] + 1, sc->iter_lo, sc->iter_hi)"),
    "role_unmasked": ("in_range(a.ctx & sc->role_mask, sc->role_lo, sc->role_hi)",
                      "in_range(a.ctx, sc->role_lo, sc->role_hi)"),
    "group_shift_ignored": ("(a.ctx >> sc->group_shift);", "(a.ctx);"),
    "mism_end_by_begin": ("stats[uint64_t(a.end_region) * ORC_RS_WIDTH + ORC_RS_MISM_AS_END] += 1;",
                          "stats[uint64_t(a.region) * ORC_RS_WIDTH + ORC_RS_MISM_AS_END] += 1;"),
    "excl_min_from_incl": ("row[ORC_RS_EXCL_MIN] = std::min(row[ORC_RS_EXCL_MIN], e);",
                           "row[ORC_RS_EXCL_MIN] = std::min(row[ORC_RS_EXCL_MIN], d);"),
    "region_mask_ignored": ("(!region_mask || region_mask[a.region] != 0)", "true"),
}

# one-line mutants of the sample attribution (argus_oracle_samples.cpp)
MUTANTS_S = {
    "end_inclusive": ("ends[ei].first <= t; ++ei)", "ends[ei].first < t; ++ei)"),
    "begin_exclusive": ("begins[bi].first <= t; ++bi)", "begins[bi].first < t; ++bi)"),
    "owner_not_required_matched": ("if (is_matched(inst[a->second])) {", "if (true) {"),
    "outermost_owner": ("for (auto a = active.rbegin(); a != active.rend(); ++a) {",
                        "for (auto a = active.begin(); a != active.end(); ++a) {"),
    "weights_ignored": ("const uint64_t w = weights ? weights[i] : 1;", "const uint64_t w = 1;"),
    "owner_parent_region": ("n_rp[uint64_t(smp[i].pc) * R + inst[owner].region] += w;",
                            "n_rp[uint64_t(smp[i].pc) * R + inst[inst[owner].parent == 0xFFFFFFFFu"
                            " ? owner : inst[owner].parent].region] += w;"),
    "entropy_sign": ("if (row[r] > 0) h -= a * std::log(a);", "if (row[r] > 0) h += a * std::log(a);"),
    "alpha_over_owners": ("const double a = row[r] > 0 ? double(row[r]) / double(T) : 0.0;",
                          "const double a = row[r] > 0 ? double(row[r]) / double(owners) : 0.0;"),
    "mhat_unweighted": ("const double term = a * metrics[k * P + p];",
                        "const double term = metrics[k * P + p];"),
    "bad_pc_not_counted": ("counters[ORC_S_N_BAD_PC] += 1;", "counters[ORC_S_N_BAD_PC] += 0;"),
    "ctx_ignored": ("auto it = inst_of.find(kv.first);", "auto it = inst_of.begin();"),
}

MUTANTS = {
    "parent_dropped": ("x.parent = stack.empty() ? kNone : stack.back();", "x.parent = kNone;"),
    "level_off_by_one": ("x.level = static_cast<uint32_t>(stack.size());",
                         "x.level = static_cast<uint32_t>(stack.size()) + 1;"),
    "excl_wrong_sign": ("excl[id] = (x.t_end - x.t_begin) - child_sum[id];",
                        "excl[id] = (x.t_end - x.t_begin) + child_sum[id];"),
    "excl_only_matched_children": ("if (is_closed(x) && x.parent != kNone)",
                                   "if (is_matched(x) && x.parent != kNone)"),
    "sort_ignores_time": ("return a.ts < b.ts;", "return false;"),
    "mismatch_counted_as_match": ("return x.end_region != kNoEnd && x.end_region == x.region;",
                                  "return x.end_region != kNoEnd;"),
    "hist_bin_shifted": ("row[ORC_RS_HIST_INCL + bit_width(d)] += 1;",
                         "row[ORC_RS_HIST_INCL + bit_width(d / 2)] += 1;"),
    "u_is_or": ("if (ca > 0 && cb > 0) U[a * K + b] += gap;",
                "if (ca > 0 || cb > 0) U[a * K + b] += gap;"),
    "q_same_class_pairs": ("Q[a * K + b] += gap * (ca * (ca - 1) / 2);",
                           "Q[a * K + b] += gap * (ca * ca / 2);"),
    "min_sentinel_zero": ("row[ORC_RS_INCL_MIN] = kNoTime;", "row[ORC_RS_INCL_MIN] = 0;"),
    "self_nested_by_end_region": ("inst[x.parent].region == x.region",
                                  "inst[x.parent].end_region == x.region"),
    "orphan_region_wrong": ("region_stats[uint64_t(r.region) * ORC_RS_WIDTH + ORC_RS_ORPHAN_END] += 1;",
                            "region_stats[ORC_RS_ORPHAN_END] += 1;"),
    "bad_region_inclusive": ("if (r.region >= num_regions) {", "if (r.region > num_regions) {"),
    "group_shift_ignored": ("(x.ctx >> group_shift)", "(x.ctx)"),
}


def run_pins(orc) -> list[str]:
    """Return the names of the pin checks that fail for oracle `orc`."""
    failures = []

    def attempt(name, fn):
        try:
            fn()
        except Exception:  # noqa: BLE001 - any failure kills the mutant
            failures.append(name)

    def hand():
        for case in load_cases():
            p = case_params(case)
            out = orc.run(records_from_rows(case["records"]), p["num_regions"],
                          p["num_classes"], p["region_class"], p["group_shift"],
                          p["num_groups"])
            np.testing.assert_array_equal(out["counters"], expected_counters(case))
            if "region_stats" in case:
                np.testing.assert_array_equal(out["region_stats"], expected_region_stats(case))
            if "instances" in case:
                assert out["instances"].tobytes() == expected_instances(case).tobytes()
                np.testing.assert_array_equal(out["instance_excl"],
                                              np.array(case["excl"], np.uint64))
            if "overlap_group" in case:
                np.testing.assert_array_equal(out["overlap_group"],
                                              np.array(case["overlap_group"], np.uint64))

    def scan():
        for seed in range(150):
            rng = np.random.default_rng(seed)
            R = 1 + seed % 5
            rec = random_malformed(rng, 48, 1 + seed % 4, R, [3, 10, 1000][seed % 3])
            out = orc.run(rec, R)
            inst, excl = scan_derivation(rec, R)
            assert out["instances"].tobytes() == inst.tobytes()
            np.testing.assert_array_equal(out["instance_excl"], excl)
            check_invariants(out, R)

    def overlap():
        for seed in range(60):
            rng = np.random.default_rng(1000 + seed)
            K, R, shift, G = 1 + seed % 3, 4, seed % 3, 1 + seed % 2
            cls = rng.integers(0, K + 1, size=R).astype(np.uint8)
            rec, ivs = random_wellformed(rng, 4, 6, R, max_depth=2, t_spread=20)
            out = orc.run(rec, R, K, cls, shift, G)
            U, Q = brute_force_overlap(ivs, K, cls, shift, G)
            np.testing.assert_array_equal(out["overlap_group"][:, 0].astype(object), U)
            np.testing.assert_array_equal(out["overlap_group"][:, 1].astype(object), Q)

    attempt("hand_traces", hand)
    attempt("depth_scan_derivation", scan)
    attempt("brute_force_overlap", overlap)
    return failures


def run_sample_pins(orc) -> list[str]:
    """The sample-attribution pins of test_oracle_samples against `orc`."""
    import test_oracle_samples as ts
    failures = []
    checks = [("hand_nested", lambda: ts.test_hand_nested_shared_helper(orc)),
              ("hand_mismatched", lambda: ts.test_hand_mismatched_innermost(orc)),
              ("hand_unclosed", lambda: ts.test_hand_unclosed_and_zero_length(orc)),
              ("hand_weights", lambda: ts.test_hand_weights_contexts_and_bad_pcs(orc)),
              ("entropy_closed_forms", lambda: ts.test_entropy_closed_forms(orc))]
    checks += [(f"brute_force_owner_{k}", (lambda k=k: ts.test_brute_force_owner(orc, k)))
               for k in range(40)]
    checks += [(f"invariants_{k}", (lambda k=k: ts.test_invariants(orc, k))) for k in range(10)]
    for name, fn in checks:
        try:
            fn()
        except Exception:  # noqa: BLE001 - any failure kills the mutant
            failures.append(name)
    return failures


@pytest.fixture(scope="module")
def mutant_dir(tmp_path_factory):
    return tmp_path_factory.mktemp("oracle_mutants")


def run_scope_pins(orc) -> list[str]:
    """The scope and ordinal pins of test_oracle_scope against `orc`."""
    import test_oracle_scope as tc
    failures = []
    checks = [("hand_ordinals", lambda: tc.test_hand_ordinals_and_window(orc)),
              ("hand_role_group_mask", lambda: tc.test_hand_role_group_and_region_mask(orc)),
              ("hand_malformed", lambda: tc.test_hand_malformed_in_scope(orc))]
    checks += [(f"brute_force_ordinal_{k}", (lambda k=k: tc.test_brute_force_ordinal(orc, k)))
               for k in range(30)]
    checks += [(f"partitions_{k}", (lambda k=k: tc.test_all_scope_and_partitions(orc, k)))
               for k in range(12)]
    for name, fn in checks:
        try:
            fn()
        except Exception:  # noqa: BLE001 - any failure kills the mutant
            failures.append(name)
    return failures


def run_probe_pins(orc) -> list[str]:
    """The probe join pins of test_oracle_probes against `orc`."""
    import test_oracle_probes as tp
    failures = []
    checks = [("hand_join", lambda: tp.test_hand_percentiles_and_join(orc)),
              ("hand_small", lambda: tp.test_hand_small_counts(orc))]
    checks += [(f"brute_force_{k}", (lambda k=k: tp.test_brute_force(orc, k))) for k in range(25)]
    for name, fn in checks:
        try:
            fn()
        except Exception:  # noqa: BLE001 - any failure kills the mutant
            failures.append(name)
    return failures


def run_handoff_pins(orc) -> list[str]:
    """The handoff pins of test_oracle_handoffs against `orc`."""
    import test_oracle_handoffs as th
    failures = []
    checks = [("hand_top", lambda: th.test_hand_top_level(orc)),
              ("hand_steps", lambda: th.test_hand_steps(orc)),
              ("hand_malformed", lambda: th.test_hand_malformed_phases(orc))]
    checks += [(f"brute_force_{k}", (lambda k=k: th.test_brute_force(orc, k))) for k in range(24)]
    checks += [(f"conservation_{k}", (lambda k=k: th.test_time_conservation(orc, k)))
               for k in range(10)]
    for name, fn in checks:
        try:
            fn()
        except Exception:  # noqa: BLE001 - any failure kills the mutant
            failures.append(name)
    return failures


def test_unmutated_oracle_passes_all_pins(oracle_mod):
    assert run_pins(oracle_mod) == []
    assert run_sample_pins(oracle_mod) == []
    assert run_scope_pins(oracle_mod) == []
    assert run_probe_pins(oracle_mod) == []
    assert run_handoff_pins(oracle_mod) == []


def _build_mutant(mutant_dir, name, target, old, new):
    src = open(target).read()
    assert src.count(old) == 1, f"mutation site for {name} not unique"
    # one file per (source, mutant): names repeat across sources, and a second
    # dlopen of a path already loaded returns the first library
    tag = f"{os.path.splitext(os.path.basename(target))[0]}_{name}"
    path = os.path.join(str(mutant_dir), f"{tag}.cpp")
    with open(path, "w") as f:
        f.write(src.replace(old, new))
    others = [x for x in SOURCES if x != target]
    inc = os.path.join(ROOT, "oracle")
    lib = os.path.join(str(mutant_dir), f"lib{tag}.so")
    subprocess.check_call(["g++", "-O1", "-std=c++17", "-ffp-contract=off", "-shared", "-fPIC",
                           "-I", inc, path, *others, "-o", lib])
    return lib


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(oracle_mod, mutant_dir, name):
    old, new = MUTANTS[name]
    orc = oracle_mod.OracleLib(_build_mutant(mutant_dir, name, SRC, old, new))
    assert run_pins(orc), f"mutant {name} survived every pin"


@pytest.mark.parametrize("name", sorted(MUTANTS_S))
def test_sample_mutant_is_caught(oracle_mod, mutant_dir, name):
    old, new = MUTANTS_S[name]
    orc = oracle_mod.OracleLib(_build_mutant(mutant_dir, name, SRC_S, old, new))
    assert run_sample_pins(orc), f"mutant {name} survived every pin"


@pytest.mark.parametrize("name", sorted(MUTANTS_C))
def test_scope_mutant_is_caught(oracle_mod, mutant_dir, name):
    old, new = MUTANTS_C[name]
    orc = oracle_mod.OracleLib(_build_mutant(mutant_dir, name, SRC_C, old, new))
    assert run_scope_pins(orc), f"mutant {name} survived every pin"


@pytest.mark.parametrize("name", sorted(MUTANTS_P))
def test_probe_mutant_is_caught(oracle_mod, mutant_dir, name):
    old, new = MUTANTS_P[name]
    orc = oracle_mod.OracleLib(_build_mutant(mutant_dir, name, SRC_P, old, new))
    assert run_probe_pins(orc), f"mutant {name} survived every pin"


@pytest.mark.parametrize("name", sorted(MUTANTS_H))
def test_handoff_mutant_is_caught(oracle_mod, mutant_dir, name):
    old, new = MUTANTS_H[name]
    orc = oracle_mod.OracleLib(_build_mutant(mutant_dir, name, SRC_H, old, new))
    assert run_handoff_pins(orc), f"mutant {name} survived every pin"
