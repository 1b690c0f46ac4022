"""Parity of the HIP path (through the C ABI) with the CPU oracle, element by
element and bit-exact: counters, per-region statistics, overlap matrices,
instances and exclusive durations.

Sizes span several sort tiles (4096) and matching tiles (2048) with ragged
tails; edge cases cover empty and all-invalid inputs, ties, orphans, unclosed
and mismatched markers, nesting deeper than a tile, contexts spanning many
tiles, keys wider than 64 bits and inputs that are out of time order inside
a context (the full sort)."""
from __future__ import annotations

import numpy as np
import pytest

from golden_util import (case_params, expected_counters, expected_instances,
                         expected_region_stats, load_cases, random_malformed,
                         random_wellformed, records_from_rows)
from gpu_util import assert_parity, gpu_run, log, oracle_run

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU in this container")
    from paper_2609_12299_amd import load_library
    load_library()  # fails loudly if the HIP library is missing
    return torch


CASES = load_cases()


@pytest.mark.parametrize("case", CASES, ids=[c["name"] for c in CASES])
def test_hand_traces(oracle_mod, case):
    log(f"[gpu] hand trace {case['name']}")
    rec = records_from_rows(case["records"])
    p = case_params(case)
    g = gpu_run(rec, p)
    np.testing.assert_array_equal(g["counters"], expected_counters(case))
    if "region_stats" in case:
        np.testing.assert_array_equal(g["region_stats"], expected_region_stats(case))
    if "instances" in case:
        assert g["instances"].tobytes() == expected_instances(case).tobytes()
        np.testing.assert_array_equal(g["instance_excl"], np.array(case["excl"], np.uint64))
    if "overlap_group" in case:
        np.testing.assert_array_equal(g["overlap_group"], np.array(case["overlap_group"], np.uint64))
    assert_parity(g, oracle_run(oracle_mod, rec, p), what=case["name"])


SIZES = [0, 1, 2, 63, 64, 65, 2047, 2048, 2049, 4095, 4096, 4097, 10007, 30001]


@pytest.mark.parametrize("ev", ["merge", "radix"])
@pytest.mark.parametrize("n", SIZES)
@pytest.mark.parametrize("n_ctx,ts_range", [(1, 1 << 40), (3, 40), (50, 1 << 20)])
def test_random_malformed(oracle_mod, n, n_ctx, ts_range, ev):
    rng = np.random.default_rng(n * 131 + n_ctx)
    R = 7
    rec = random_malformed(rng, n, n_ctx, R, ts_range)
    cls = rng.integers(0, 4, size=R).astype(np.uint8)
    p = dict(num_regions=R, num_classes=3, region_class=cls, group_shift=1, num_groups=20)
    log(f"[gpu] random malformed n={n} ctx={n_ctx} ts_range={ts_range} events={ev}")
    g = gpu_run(rec, p, force_event=ev == "radix", with_plan=True)
    if int(g["counters"][1]) > 0:
        assert g["_plan"]["ev_merge"] == (1 if ev == "merge" else 0)
    assert_parity(g, oracle_run(oracle_mod, rec, p), what=f"n={n}")


def _nested_contexts(rng, ctx_sizes, R, t_spread, ts_base=0):
    """Well-formed nested regions in each context, `size` records each (even),
    timestamps overlapping across contexts, rows shuffled."""
    rows = []
    for c, size in ctx_sizes:
        t = ts_base + int(rng.integers(0, t_spread))
        stack, left = [], size
        while left > 0:
            if stack and (len(stack) >= left or len(stack) >= 6 or rng.random() < 0.45):
                rows.append((t, c, stack.pop(), 2))
            else:
                r = int(rng.integers(0, R))
                stack.append(r)
                rows.append((t, c, r, 1))
            left -= 1
            t += int(rng.integers(0, 3 * t_spread // max(size, 1) + 2))
    order = rng.permutation(len(rows))
    return records_from_rows([rows[i] for i in order])


@pytest.mark.parametrize("shift,G", [(5, 3), (3, 100), (32, 1)])
def test_merge_many_small_contexts(oracle_mod, shift, G):
    """Hundreds of tiny contexts per group (segments far smaller than a merge
    tile, many segments per round), groups beyond G present."""
    rng = np.random.default_rng(shift * 7 + G)
    ctxs = sorted(rng.choice(1 << 8, size=150, replace=False).tolist())
    rec = _nested_contexts(rng, [(c, int(rng.integers(1, 6)) * 2) for c in ctxs], 5, 1 << 40)
    p = dict(num_regions=5, num_classes=3, region_class=np.array([0, 1, 2, 1, 7], np.uint8),
             group_shift=shift, num_groups=G)
    log(f"[gpu] merge: many small contexts shift={shift} G={G} n={len(rec)}")
    g = gpu_run(rec, p, with_plan=True)
    assert g["_plan"]["ev_merge"] == 1
    assert_parity(g, oracle_run(oracle_mod, rec, p))


def test_merge_skewed_contexts(oracle_mod):
    """One group: a context spanning many merge tiles next to contexts of a
    few records, and eight context bits (0..7) merged in four four-way
    passes."""
    rng = np.random.default_rng(77)
    sizes = [(0, 40000), (1, 2), (2, 4), (4, 30000), (8, 6), (16, 9000), (32, 2), (64, 12),
             (128, 5000)]
    rec = _nested_contexts(rng, sizes, 6, 1 << 56)
    p = dict(num_regions=6, num_classes=2, region_class=np.array([0, 1, 0, 1, 5, 0], np.uint8),
             group_shift=32, num_groups=1)
    log(f"[gpu] merge: skewed contexts n={len(rec)}")
    g = gpu_run(rec, p, with_plan=True)
    assert g["_plan"]["ev_merge"] == 1 and g["_plan"]["merge_rounds"] == 4
    assert_parity(g, oracle_run(oracle_mod, rec, p))


@pytest.mark.parametrize("case", ["odd_bits", "empty_runs", "five_bits", "ties"])
def test_merge_four_way(oracle_mod, case):
    """Four-way passes: three context bits (a four-way pass, then a two-way
    last pass), segments of a four-way pass with empty runs in the middle
    and at the end (classes 0 and 3 only; 0 and 1 only), five bits (two
    stored four-way passes), and runs of equal timestamps across the four
    runs of a segment, each over several tiles."""
    rng = np.random.default_rng(["odd_bits", "empty_runs", "five_bits", "ties"].index(case) + 101)
    spread, passes = 1 << 36, None
    if case == "odd_bits":
        sizes = [(0, 9000), (1, 3000), (2, 700), (3, 12000), (4, 5), (5, 2), (6, 8000), (7, 40)]
        shift, passes = 3, 2
    elif case == "empty_runs":
        # bits 0 and 1 in one pass: segment {0, 1} has runs 2, 3 empty,
        # segment {4, 7} runs 1, 2; bit 2 in the last pass
        sizes = [(c + 8 * g, 2 * int(rng.integers(1, 4500))) for g in range(3) for c in (0, 1, 4, 7)]
        shift, passes = 3, 2
    elif case == "five_bits":
        sizes = [(c, 2 * int(rng.integers(1, 2000))) for c in range(32) if rng.random() < 0.8]
        sizes[len(sizes) // 2] = (sizes[len(sizes) // 2][0], 30000)
        shift, passes = 5, 3
    else:
        sizes = [(c, 6000) for c in range(4)] + [(c, 3000) for c in range(4, 16)]
        spread, shift, passes = 300, 4, 2
    rec = _nested_contexts(rng, sizes, 6, spread)
    p = dict(num_regions=6, num_classes=3, region_class=np.array([0, 1, 2, 1, 0, 9], np.uint8),
             group_shift=shift, num_groups=1 << (12 - shift) if shift < 12 else 1)
    log(f"[gpu] merge four-way: {case} n={len(rec)}")
    g = gpu_run(rec, p, with_plan=True)
    assert g["_plan"]["ev_merge"] == 1
    if passes is not None:
        assert g["_plan"]["merge_rounds"] == passes
    assert_parity(g, oracle_run(oracle_mod, rec, p))


@pytest.mark.parametrize("why", ["bits", "rounds"])
def test_event_radix_fallback(oracle_mod, why):
    """Where merging does not apply the radix sort orders the events: the
    event word would need more than 64 bits, or merging would take more
    rounds than the sort takes passes."""
    rng = np.random.default_rng(9)
    if why == "bits":
        sizes = [(c, 400) for c in range(0, 64, 3)]
        rec = _nested_contexts(rng, sizes, 4, 1 << 61)
        p = dict(num_regions=4, num_classes=2, region_class=np.array([0, 1, 1, 0], np.uint8),
                 group_shift=2, num_groups=1 << 12)
    else:
        sizes = [(c, 40) for c in rng.choice(1 << 12, size=300, replace=False).tolist()]
        rec = _nested_contexts(rng, sizes, 4, 200)
        p = dict(num_regions=4, num_classes=2, region_class=np.array([0, 1, 1, 0], np.uint8),
                 group_shift=12, num_groups=1)
    log(f"[gpu] event radix fallback ({why}) n={len(rec)}")
    g = gpu_run(rec, p, with_plan=True)
    assert g["_plan"]["ev_merge"] == 0
    assert_parity(g, oracle_run(oracle_mod, rec, p))


@pytest.mark.parametrize("force_full", [False, True])
@pytest.mark.parametrize("seed", [0, 1])
def test_random_wellformed(oracle_mod, seed, force_full):
    rng = np.random.default_rng(100 + seed)
    rec, _ = random_wellformed(rng, 40, 300, 6, max_depth=5, t_spread=9)
    cls = np.array([0, 1, 2, 0, 255, 1], np.uint8)
    p = dict(num_regions=6, num_classes=3, region_class=cls, group_shift=3, num_groups=5)
    log(f"[gpu] random wellformed seed={seed} force_full={force_full} n={len(rec)}")
    assert_parity(gpu_run(rec, p, force_full=force_full), oracle_run(oracle_mod, rec, p))


def test_nesting_deeper_than_a_tile(oracle_mod):
    rows, t = [], 0
    for ctx in (5, 6):
        for k in range(5000):
            rows.append((t, ctx, k % 9, 1))
            t += 1
        for k in reversed(range(5000)):
            rows.append((t, ctx, k % 9 if k % 97 else (k + 1) % 9, 2))
            t += 1
    rows.append((t, 6, 3, 2))  # an orphan after the context unwinds
    rec = records_from_rows(rows)
    p = dict(num_regions=9, num_classes=2, region_class=np.array([0, 1] * 4 + [9], np.uint8),
             group_shift=0, num_groups=8)
    log("[gpu] nesting deeper than a tile")
    assert_parity(gpu_run(rec, p), oracle_run(oracle_mod, rec, p))


@pytest.mark.parametrize("drift", ["up", "down", "balanced"])
def test_long_context_with_drift(oracle_mod, drift):
    """One context over ~25 tiles whose depth drifts (duplicate BEGINs or orphan
    ENDs), so pairs, parents and child sums cross many tiles."""
    rng = np.random.default_rng({"up": 1, "down": 2, "balanced": 3}[drift])
    p_begin = {"up": 0.52, "down": 0.48, "balanced": 0.5}[drift]
    n = 50000
    kinds = np.where(rng.random(n) < p_begin, 1, 2)
    ts = np.cumsum(rng.integers(0, 4, size=n))  # zero gaps give ties
    regs = rng.integers(0, 5, size=n)
    ctx = np.full(n, 11)
    ctx[rng.random(n) < 0.01] = 12
    rows = list(zip(ts.tolist(), ctx.tolist(), regs.tolist(), kinds.tolist()))
    rec = records_from_rows(rows)
    p = dict(num_regions=5, num_classes=2, region_class=np.array([0, 1, 0, 1, 0], np.uint8),
             group_shift=1, num_groups=7)
    log(f"[gpu] long context drift={drift}")
    assert_parity(gpu_run(rec, p), oracle_run(oracle_mod, rec, p))


def test_wide_keys(oracle_mod):
    """Context keys spread over 32 bits and a 40-bit time span: the packed
    (ctx, ts) key needs more than 64 bits."""
    rng = np.random.default_rng(5)
    rows = []
    for c in rng.integers(0, 1 << 32, size=64, dtype=np.uint64).tolist():
        t = int(rng.integers(0, 1 << 40))
        depth, stack = 0, []
        for k in range(120):
            if depth == 0 or (depth < 4 and rng.random() < 0.5):
                r = int(rng.integers(0, 6))
                stack.append(r)
                rows.append((t, c, r, 1))
                depth += 1
            else:
                rows.append((t, c, stack.pop(), 2))
                depth -= 1
            t += int(rng.integers(1, 1 << 20))
    rng.shuffle(rows)
    rec = records_from_rows(rows)
    p = dict(num_regions=6, num_classes=2, region_class=np.array([0, 1, 0, 1, 0, 1], np.uint8),
             group_shift=24, num_groups=256)
    log("[gpu] wide keys")
    assert_parity(gpu_run(rec, p), oracle_run(oracle_mod, rec, p))


@pytest.mark.parametrize("force_full", [False, True])
@pytest.mark.parametrize("cfg,kw", [(1, {}), (2, dict(blocks=4)), (3, dict(blocks=2)),
                                    (4, dict(blocks=4)), (5, dict(blocks=16, size=1 << 20))])
def test_workload_shapes_scaled(oracle_mod, tracegen_mod, cfg, kw, force_full):
    d = tracegen_mod.generate(cfg, **kw)
    p = {k: d[k] for k in ("num_regions", "num_classes", "region_class", "group_shift", "num_groups")}
    log(f"[gpu] config {cfg} {kw} force_full={force_full} n={len(d['records'])}")
    assert_parity(gpu_run(d["records"], p, force_full=force_full),
                  oracle_run(oracle_mod, d["records"], p), what=f"cfg{cfg}")


@pytest.mark.parametrize("cfg,kw", [(2, dict(blocks=4)), (3, dict(blocks=2)), (4, dict(blocks=4)),
                                    (5, dict(blocks=16, size=1 << 20))])
def test_workload_shapes_event_radix(oracle_mod, tracegen_mod, cfg, kw):
    """The event radix sort on the workload shapes (merging is the default)."""
    d = tracegen_mod.generate(cfg, **kw)
    p = {k: d[k] for k in ("num_regions", "num_classes", "region_class", "group_shift", "num_groups")}
    log(f"[gpu] config {cfg} {kw} event radix n={len(d['records'])}")
    g = gpu_run(d["records"], p, force_event=True, with_plan=True)
    assert g["_plan"]["ev_merge"] == 0
    assert_parity(g, oracle_run(oracle_mod, d["records"], p), what=f"cfg{cfg}")


def test_determinism_and_stream(oracle_mod, tracegen_mod, gpu):
    d = tracegen_mod.generate(5, blocks=8, size=1 << 18)
    p = {k: d[k] for k in ("num_regions", "num_classes", "region_class", "group_shift", "num_groups")}
    log("[gpu] determinism, non-default stream")
    s = gpu.cuda.Stream()
    a, b = gpu_run(d["records"], p, stream=s, repeat=2)
    for k in a:
        np.testing.assert_array_equal(a[k], b[k])
    assert_parity(a, oracle_run(oracle_mod, d["records"], p))


def test_without_instance_outputs(oracle_mod, tracegen_mod):
    d = tracegen_mod.generate(3, blocks=1)
    p = {k: d[k] for k in ("num_regions", "num_classes", "region_class", "group_shift", "num_groups")}
    log("[gpu] statistics only (instances in the workspace)")
    g = gpu_run(d["records"], p, instances=False)
    assert_parity(g, oracle_run(oracle_mod, d["records"], p, instances=False), instances=False)


@pytest.mark.parametrize("depth", [700, 1500])
def test_enclosing_levels_beyond_lds(oracle_mod, depth):
    """A tile that starts `depth` levels deep, closes a child of an instance
    opened in an earlier tile, and then unwinds every level: the child sums
    of enclosing instances more than 512 levels above the tile's low point
    take the global-memory path of the matching kernel."""
    rows, t = [], 0
    for k in range(depth):
        rows.append((t, 7, k % 5, 1))
        t += 1
    # pairs at the top until the next record starts a matching tile
    while len(rows) < 2048:
        rows.append((t, 7, 1, 1))
        rows.append((t + 3, 7, 1, 2))
        t += 5
    rows = rows[:2048]
    for j in range(6):  # children of the level depth-1 instance, in the new tile
        rows.append((t, 7, 2, 1))
        rows.append((t + 7, 7, 2, 2))
        t += 9
    for k in reversed(range(depth)):
        rows.append((t, 7, k % 5, 2))
        t += 2
    rec = records_from_rows(rows)
    p = dict(num_regions=5, num_classes=2, region_class=np.array([0, 1, 0, 1, 0], np.uint8),
             group_shift=0, num_groups=16)
    log(f"[gpu] enclosing levels beyond LDS depth={depth}")
    assert_parity(gpu_run(rec, p), oracle_run(oracle_mod, rec, p))


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5, 6, 7, 8])
@pytest.mark.parametrize("span", ["narrow", "wide"])
def test_overlap_every_class_count(oracle_mod, k, span):
    """Class-overlap sums for every number of classes, with groups of several
    contexts (merged runs), tiles spanning less and more than 2^32 cycles,
    and unclassified regions."""
    rng = np.random.default_rng(100 * k + (span == "wide"))
    R = 12
    cls = np.array([(r % (k + 1)) if (r % (k + 1)) < k else 0xFF for r in range(R)], np.uint8)
    rows = []
    gap_hi = 1 << 34 if span == "wide" else 64
    for ctx in range(24):
        t = int(rng.integers(0, 1 << 20))
        stack = []
        for _ in range(int(rng.integers(200, 900))):
            if stack and (len(stack) > 5 or rng.random() < 0.45):
                rows.append((t, ctx, stack.pop(), 2))
            else:
                r = int(rng.integers(0, R))
                stack.append(r)
                rows.append((t, ctx, r, 1))
            t += int(rng.integers(0, gap_hi)) if rng.random() < 0.05 else int(rng.integers(0, 9))
    rec = records_from_rows(rows)
    rng.shuffle(rec)
    p = dict(num_regions=R, num_classes=k, region_class=cls, group_shift=2, num_groups=6)
    log(f"[gpu] overlap k={k} span={span} n={len(rec)}")
    assert_parity(gpu_run(rec, p), oracle_run(oracle_mod, rec, p))


def _chunked(rng, n_ctx, per_ctx, chunk, ts_step=7, unsorted=0, bad=0.0, ctx_base=0):
    """Records of n_ctx contexts interleaved `chunk` at a time (trace buffers
    written per warp), optionally with `unsorted` records moved back in time
    and a fraction `bad` of invalid kinds."""
    rows = []
    for c in range(n_ctx):
        t, depth = int(rng.integers(0, 1 << 30)), 0
        cr = []
        for _ in range(per_ctx):
            if depth and rng.random() < 0.5:
                cr.append((t, ctx_base + c, int(rng.integers(0, 6)), 2))
                depth -= 1
            else:
                cr.append((t, ctx_base + c, int(rng.integers(0, 6)), 1))
                depth += 1
            t += int(rng.integers(1, ts_step))
        for _ in range(unsorted):
            k = int(rng.integers(1, len(cr)))
            ts, cx, r, kd = cr[k]
            cr[k] = (max(0, ts - 50), cx, r, kd)
        rows.append(cr)
    out, left = [], True
    pos = [0] * n_ctx
    while left:
        left = False
        for c in range(n_ctx):
            take = rows[c][pos[c]:pos[c] + chunk]
            pos[c] += len(take)
            out.extend(take)
            left |= pos[c] < len(rows[c])
    rec = records_from_rows(out)
    if bad:
        mask = rng.random(len(rec)) < bad
        rec[mask, 14] = 3  # no such kind
    return rec


@pytest.mark.parametrize("radix", [False, True])
@pytest.mark.parametrize("shape", ["aligned", "ragged", "one_pass_unsorted", "two_pass_unsorted",
                                   "invalid_inside", "all_invalid_chunks", "short_runs"])
def test_context_sort_paths(oracle_mod, shape, radix):
    """The context sort over runs (chunked inputs) and the radix passes over
    records give identical results, including when the run path is followed
    by the full sort (with one and with two run passes before it)."""
    seeds = {"aligned": 1, "ragged": 2, "one_pass_unsorted": 3, "two_pass_unsorted": 4,
             "invalid_inside": 5, "all_invalid_chunks": 6, "short_runs": 7}
    rng = np.random.default_rng(seeds[shape])
    if shape == "aligned":
        rec = _chunked(rng, 40, 1024, 256)
    elif shape == "ragged":
        rec = _chunked(rng, 37, int(rng.integers(300, 900)), 97)
    elif shape == "one_pass_unsorted":  # contexts < 256: one context digit
        rec = _chunked(rng, 200, 300, 64, unsorted=3)
    elif shape == "two_pass_unsorted":  # contexts spread over two digits
        rec = _chunked(rng, 60, 400, 128, unsorted=2, ctx_base=250)
    elif shape == "invalid_inside":
        rec = _chunked(rng, 30, 800, 256, bad=0.02)
    elif shape == "all_invalid_chunks":
        rec = _chunked(rng, 30, 800, 256)
        rec[256:1024, 14] = 0
        rec[5000:5300, 12] = 0xFF  # bad region (>= R)
    else:  # runs too short for the run path: the radix passes either way
        rec = _chunked(rng, 64, 200, 3)
    p = dict(num_regions=6, num_classes=3, region_class=np.array([0, 1, 2, 0, 1, 0xFF], np.uint8),
             group_shift=2, num_groups=64)
    log(f"[gpu] context sort shape={shape} radix={radix} n={len(rec)}")
    g = gpu_run(rec, p, force_radix=radix, with_plan=True)
    plan = g.pop("_plan")
    if radix or shape == "short_runs":
        assert plan["runs"] == 0
    else:
        assert plan["runs"] == 1
    if "unsorted" in shape:
        assert plan["unsorted"] == 1
    assert_parity(g, oracle_run(oracle_mod, rec, p), what=shape)


@pytest.mark.parametrize("R", [1000, 1500, 5000])
@pytest.mark.parametrize("sort", ["runs", "radix"])
def test_many_regions(oracle_mod, R, sort):
    """Region counts on both sides of the statistics' and class tables' LDS
    limits: per-block partial statistics (1000), statistics in global memory
    (1500, 5000) and class tables read from global memory (5000), with the
    histograms in several slices."""
    rng = np.random.default_rng(R + (sort == "radix"))
    rec = _chunked(rng, 24, 1500, 256, bad=0.01)
    regions = rng.integers(0, R + R // 50, size=len(rec))  # a few out of range
    rec[:, 12] = (regions & 0xFF).astype(np.uint8)
    rec[:, 13] = (regions >> 8).astype(np.uint8)
    cls = rng.integers(0, 5, size=R).astype(np.uint8)  # class 4: none (K = 4)
    p = dict(num_regions=R, num_classes=4, region_class=cls, group_shift=2, num_groups=5)
    log(f"[gpu] many regions R={R} sort={sort} n={len(rec)}")
    assert_parity(gpu_run(rec, p, force_radix=sort == "radix"), oracle_run(oracle_mod, rec, p))


def test_timing_filter(oracle_mod, tracegen_mod):
    """Per-launch timing: every launch without a filter, only the named
    step's launches with one; results unchanged either way."""
    import torch

    from paper_2609_12299_amd import RegionAttribution, to_host
    d = tracegen_mod.generate(1, size=1 << 14, threads=2)
    p = {k: d[k] for k in ("num_regions", "num_classes", "region_class", "group_shift", "num_groups")}
    rec_u8 = d["records"]
    n = rec_u8.shape[0]
    ra = RegionAttribution(p["num_regions"], p["num_classes"], p["region_class"], p["group_shift"],
                           p["num_groups"], max_records=n, instances=True, instance_excl=True)
    rec = torch.from_numpy(np.ascontiguousarray(rec_u8).reshape(-1)).to("cuda")
    log("[gpu] timing filter")
    try:
        ra.set_timing(True)
        ra.run(rec)
        all_times = ra.kernel_times()
        names = [k for k, _ in all_times]
        assert "match" in names and "agg" in names and len(names) > 10
        assert all(ms >= 0.0 for _, ms in all_times)
        ra.set_timing_filter("match")
        out = ra.run(rec)
        out2 = ra.run(rec)
        torch.cuda.synchronize()
        only = ra.kernel_times()
        assert [k for k, _ in only] == ["match", "match"]
        assert all(ms > 0.0 for _, ms in only)
        ra.set_timing_filter(None)
        ra.set_timing(False)
        assert_parity(to_host(out), oracle_run(oracle_mod, rec_u8, p), what="filtered timing")
        assert_parity(to_host(out2), oracle_run(oracle_mod, rec_u8, p), what="filtered timing, second run")
    finally:
        ra.close()
