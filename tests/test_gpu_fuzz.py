"""Fuzz: about a thousand small random traces, each compared with the
oracle bit for bit, the run stopping at the first mismatch.  The traces mix
every anomaly the definitions name (bad kinds, bad regions, ties in (ctx,
ts), orphan ENDs, mismatched and unclosed BEGINs, deep nesting, contexts
that straddle the 2048-record tiles) and vary the overlap settings (classes,
group shift, groups), the event ordering (merge and radix sort) and the
context sort (over runs and over records)."""
from __future__ import annotations

import numpy as np
import pytest

from golden_util import RECORD_DTYPE
from gpu_util import log

pytestmark = pytest.mark.gpu

CASES = 1000


def random_trace(rng):
    n = int(rng.choice([rng.integers(0, 64), rng.integers(64, 1500), rng.integers(1500, 6000)]))
    n_ctx = int(rng.integers(1, 40))
    R = int(rng.integers(1, 20))
    rec = np.zeros(n, RECORD_DTYPE)
    ctx = rng.integers(0, n_ctx, size=n).astype(np.uint32) * np.uint32(rng.integers(1, 5))
    if rng.random() < 0.5:  # long runs of one context, as trace buffers have
        ctx = np.sort(ctx, kind="stable")
    rec["ctx_key"] = ctx
    spread = int(rng.choice([4, 50, 1 << 20, 1 << 40]))
    rec["ts"] = rng.integers(0, spread, size=n).astype(np.uint64)
    if rng.random() < 0.5:  # time order inside each context (a well-behaved buffer)
        rec["ts"] = np.sort(rec["ts"])
    p_begin = float(rng.uniform(0.3, 0.7))  # drift: deep nesting or many orphans
    kind = np.where(rng.random(n) < p_begin, 1, 2).astype(np.uint8)
    bad = rng.random(n) < float(rng.choice([0.0, 0.02]))
    kind[bad] = rng.choice(np.array([0, 3, 255], np.uint8), size=int(bad.sum()))
    rec["kind"] = kind
    rec["region_id"] = rng.integers(0, R + (1 if rng.random() < 0.3 else 0), size=n)
    K = int(rng.integers(0, 5))
    p = dict(num_regions=R, num_classes=K,
             region_class=rng.integers(0, K + 1, size=R).astype(np.uint8) if K else None,
             group_shift=int(rng.integers(0, 4)), num_groups=int(rng.integers(1, 12)) if K else 0)
    return rec.view(np.uint8).reshape(n, 16), p


def test_fuzz_random_traces(oracle_mod):
    import torch

    from gpu_util import assert_parity
    from paper_2609_12299_amd import RegionAttribution, to_host
    rng = np.random.default_rng(20260)
    handles = {}
    for case in range(CASES):
        rec_u8, p = random_trace(rng)
        flags = (bool(case % 3 == 1), bool(case % 5 == 2), bool(case % 7 == 3))  # full sort, event sort, record radix
        key = (p["num_regions"], p["num_classes"], p["group_shift"], p["num_groups"],
               None if p["region_class"] is None else p["region_class"].tobytes(), flags)
        ra = handles.get(key)
        if ra is None:
            ra = RegionAttribution(p["num_regions"], p["num_classes"], p["region_class"],
                                   p["group_shift"], p["num_groups"], max_records=8192,
                                   force_full_sort=flags[0], force_event_sort=flags[1],
                                   force_record_radix=flags[2])
            handles[key] = ra
        n = rec_u8.shape[0]
        rec = torch.from_numpy(np.ascontiguousarray(rec_u8).reshape(-1)).to("cuda")
        out = ra.run(rec)
        torch.cuda.synchronize()
        g = to_host(out)
        o = oracle_mod.run(rec_u8, p["num_regions"], p["num_classes"], p["region_class"],
                           p["group_shift"], p["num_groups"])
        try:
            assert_parity(g, o, what=f"fuzz case {case}")
        except AssertionError:
            log(f"[gpu] fuzz case {case} failed: n={n} params={p} flags={flags}")
            raise
        if case % 200 == 0:
            log(f"[gpu] fuzz: {case} cases compared")
    for ra in handles.values():
        ra.close()
