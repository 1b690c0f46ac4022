"""Helpers shared by the oracle pins and the GPU parity tests: loading the
hand-built golden traces and building small random traces.  No attribution
arithmetic lives here."""
from __future__ import annotations

import json
import os

import numpy as np

U64_MAX = (1 << 64) - 1
NONE32 = 0xFFFFFFFF
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "hand_traces.json")

COUNTER_NAMES = [
    "n_records", "n_valid", "n_bad_kind", "n_bad_region", "n_begin", "n_end",
    "ts_min", "ts_max", "n_ctx", "n_matched", "n_mismatched", "n_unclosed",
    "n_orphan_end", "n_self_nested", "max_level", "n_overlap_skipped",
    "ctx_min", "ctx_max",
]
RS_FIELDS = dict(count=0, incl_sum=1, excl_sum=2, incl_min=3, incl_max=4, excl_min=5,
                 excl_max=6, unclosed=7, orphan_end=8, mism_as_begin=9, mism_as_end=10,
                 self_nested=11)
RS_HIST_INCL, RS_HIST_EXCL, RS_WIDTH = 12, 77, 142

RECORD_DTYPE = np.dtype([("ts", "<u8"), ("ctx_key", "<u4"), ("region_id", "<u2"),
                         ("kind", "u1"), ("pad", "u1")])
INSTANCE_DTYPE = np.dtype([
    ("t_begin", "<u8"), ("t_end", "<u8"), ("ctx_key", "<u4"), ("parent", "<u4"),
    ("level", "<u4"), ("region_id", "<u2"), ("end_region_id", "<u2"),
])


def load_cases():
    with open(GOLDEN) as f:
        return json.load(f)["cases"]


def records_from_rows(rows) -> np.ndarray:
    a = np.zeros(len(rows), RECORD_DTYPE)
    for i, (ts, ctx, region, kind) in enumerate(rows):
        a[i] = (ts, ctx, region, kind, 0)
    return a.view(np.uint8).reshape(len(rows), 16)


def case_params(case):
    R = case["num_regions"]
    K = case.get("num_classes", 0)
    cls = np.array(case.get("region_class", [255] * R), np.uint8)
    return dict(num_regions=R, num_classes=K, region_class=cls,
                group_shift=case.get("group_shift", 0), num_groups=case.get("num_groups", 0))


def expected_counters(case) -> np.ndarray:
    c = np.zeros(32, np.uint64)
    c[COUNTER_NAMES.index("ts_min")] = U64_MAX
    c[COUNTER_NAMES.index("ctx_min")] = U64_MAX
    for k, v in case["counters"].items():
        c[COUNTER_NAMES.index(k)] = v
    return c


def expected_region_stats(case) -> np.ndarray:
    R = case["num_regions"]
    rs = np.zeros((R, RS_WIDTH), np.uint64)
    rs[:, RS_FIELDS["incl_min"]] = U64_MAX
    rs[:, RS_FIELDS["excl_min"]] = U64_MAX
    for r, fields in case.get("region_stats", {}).items():
        r = int(r)
        for k, v in fields.items():
            if k == "hist_incl":
                for b, cnt in v.items():
                    rs[r, RS_HIST_INCL + int(b)] = cnt
            elif k == "hist_excl":
                for b, cnt in v.items():
                    rs[r, RS_HIST_EXCL + int(b)] = cnt
            else:
                rs[r, RS_FIELDS[k]] = v
    return rs


def expected_instances(case) -> np.ndarray:
    rows = case["instances"]
    a = np.zeros(len(rows), INSTANCE_DTYPE)
    for i, row in enumerate(rows):
        a[i] = tuple(row)
    return a


# ---------------------------------------------------------------- random traces

def random_wellformed(rng: np.random.Generator, n_ctx: int, per_ctx_pairs: int, R: int,
                      max_depth: int = 4, ctx_keys=None, t_spread: int = 5):
    """A random well-formed nested trace and the intervals it contains.

    Returns (records uint8 [N,16] in a shuffled input order,
             intervals list of (ctx, region, t_begin, t_end, level)).
    Timestamps strictly increase inside a context, so (ctx, ts) keys are
    distinct and the input order does not matter.
    """
    rows, ivs = [], []
    keys = ctx_keys if ctx_keys is not None else list(range(n_ctx))
    for ctx in keys:
        t = int(rng.integers(0, 50))
        stack = []
        opened = 0
        while opened < per_ctx_pairs or stack:
            can_open = opened < per_ctx_pairs and len(stack) < max_depth
            if can_open and (not stack or rng.random() < 0.5):
                reg = int(rng.integers(0, R))
                stack.append((reg, t, len(stack)))
                rows.append((t, ctx, reg, 1))
                opened += 1
            else:
                reg, t0, lvl = stack.pop()
                rows.append((t, ctx, reg, 2))
                ivs.append((ctx, reg, t0, t, lvl))
            t += int(rng.integers(1, t_spread + 1))
    perm = rng.permutation(len(rows))
    rows = [rows[i] for i in perm]
    return records_from_rows(rows), ivs


def random_malformed(rng: np.random.Generator, n: int, n_ctx: int, R: int, ts_range: int,
                     p_bad: float = 0.1):
    """Random records: BEGIN/END of random regions at random times (ties are
    likely), with a few bad kinds and bad regions mixed in."""
    rows = []
    for _ in range(n):
        ts = int(rng.integers(0, ts_range))
        ctx = int(rng.integers(0, n_ctx))
        u = rng.random()
        if u < p_bad / 2:
            kind = int(rng.choice([0, 3, 7, 255]))
            reg = int(rng.integers(0, R))
        elif u < p_bad:
            kind = int(rng.integers(1, 3))
            reg = int(rng.integers(R, R + 3))
        else:
            kind = int(rng.integers(1, 3))
            reg = int(rng.integers(0, R))
        rows.append((ts, ctx, reg, kind))
    return records_from_rows(rows)
