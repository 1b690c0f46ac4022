"""PC-sample attribution on the GPU (argus_attr_samples) against the oracle.

The GPU side attributes samples to the instance array that argus_attr_run
wrote on the device (its instance count read on the device from the run's
counters); the oracle side attributes them to the oracle's own instances.
Integers (counts, totals, owners, counters) must be identical, and so must
alpha (one correctly rounded division each) and m_hat (a fixed order of
rounded operations).  H(p) goes through the device logarithm and a
different summation order, so it is compared within the bound derived from
its arithmetic: every term -alpha log alpha is >= 0, each side's error is at
most (owners + 4) ulp-units of eps = 2^-53 times H, so the two agree within
2 (owners + 4) eps H (plus 1e-300 for H == 0).
"""
from __future__ import annotations

import numpy as np
import pytest

from golden_util import random_malformed, records_from_rows
from gpu_util import log

pytestmark = pytest.mark.gpu

EPS = 2.0 ** -53


def run_both(oracle_mod, rec_u8, R, samples, P, weights=None, metrics=None, K=0, cls=None,
             shift=0, G=0):
    import torch

    from paper_2609_12299_amd import RegionAttribution, attribute_samples
    n = rec_u8.shape[0]
    ra = RegionAttribution(R, K, cls, shift, G, max_records=max(n, 1))
    rec = torch.from_numpy(np.ascontiguousarray(rec_u8).reshape(-1)).to("cuda")
    out = ra.run(rec)
    smp = torch.from_numpy(np.ascontiguousarray(samples).view(np.uint8).reshape(-1)).to("cuda")
    w = torch.from_numpy(np.ascontiguousarray(weights)).to("cuda") if weights is not None else None
    m = torch.from_numpy(np.ascontiguousarray(metrics)).to("cuda") if metrics is not None else None
    g = attribute_samples(out["instances"], out["counters"][4:5], smp, R, P, weights=w, metrics=m)
    torch.cuda.synchronize()
    g = {k: v.cpu().numpy() for k, v in g.items()}
    ra.close()
    oi = oracle_mod.run(rec_u8, R, K, cls, shift, G)["instances"]
    o = oracle_mod.samples(oi, samples, R, P, weights=weights, metrics=metrics)
    return g, o


def assert_samples_parity(g, o, what=""):
    np.testing.assert_array_equal(g["counters"][:7], o["counters"][:7], err_msg=f"{what}: counters")
    assert int(g["counters"][7]) == 0, f"{what}: samples owned by out-of-range regions"
    for k in ("n", "pc_total", "pc_owners", "region_total"):
        np.testing.assert_array_equal(g[k], o[k], err_msg=f"{what}: {k}")
    for k in ("alpha", "mhat"):
        a, b = g[k], o[k]
        assert a.shape == b.shape and a.tobytes() == b.tobytes(), \
            f"{what}: {k} not bit-identical (max |diff| {np.max(np.abs(a - b)) if a.size else 0})"
    tol = 2 * (o["pc_owners"].astype(np.float64) + 4) * EPS * o["entropy"] + 1e-300
    bad = np.abs(g["entropy"] - o["entropy"]) > tol
    assert not bad.any(), f"{what}: entropy off at {np.nonzero(bad)[0][:5]}"


def _samples(rows):
    from paper_2609_12299_amd import SAMPLE_DTYPE
    s = np.zeros(len(rows), SAMPLE_DTYPE)
    for i, r in enumerate(rows):
        s[i] = r
    return s


def test_hand_trace(oracle_mod):
    rec = records_from_rows([(0, 0, 0, 1), (20, 0, 1, 1), (50, 0, 1, 2), (100, 0, 0, 2)])
    smp = _samples([(10, 0, 7), (30, 0, 7), (40, 0, 7), (60, 0, 7), (0, 0, 3), (25, 0, 3),
                    (26, 0, 3), (100, 0, 3)])
    m = np.zeros((1, 8))
    m[0, 3], m[0, 7] = 6.0, 10.0
    g, o = run_both(oracle_mod, rec, 2, smp, 8, metrics=m)
    assert g["n"][7].tolist() == [2, 2] and g["n"][3].tolist() == [1, 2]
    assert_samples_parity(g, o, "hand")


@pytest.mark.parametrize("n,ns,n_ctx,R,P,tr", [
    (0, 100, 3, 3, 5, 50), (7, 0, 2, 2, 3, 10), (300, 2000, 4, 5, 7, 200),
    (2049, 5000, 3, 6, 40, 3000), (30001, 70001, 17, 9, 300, 40000),
    (100000, 300000, 64, 40, 1000, 1 << 20),
    # many instances over a table of 3 PCs x 2 regions
    (5000, 3000, 3, 2, 3, 4000)])
def test_random_malformed(oracle_mod, n, ns, n_ctx, R, P, tr):
    rng = np.random.default_rng(n + ns)
    rec = random_malformed(rng, n, n_ctx, R, tr)
    from paper_2609_12299_amd import SAMPLE_DTYPE
    smp = np.zeros(ns, SAMPLE_DTYPE)
    smp["ts"] = rng.integers(0, tr + 5, size=ns)
    smp["ctx_key"] = rng.integers(0, n_ctx + 1, size=ns)
    smp["pc"] = rng.integers(0, P + 1, size=ns)
    w = rng.integers(1, 1000, size=ns).astype(np.uint32)
    m = rng.normal(size=(3, P)) * 1e3
    log(f"[gpu] samples random: n={n} samples={ns} R={R} P={P}")
    g, o = run_both(oracle_mod, rec, R, smp, P, weights=w, metrics=m)
    assert_samples_parity(g, o, f"random n={n}")


def test_no_metrics_many_pcs(oracle_mod):
    """No PC metrics (M = 0): counts, alpha, entropy and region totals only,
    over 5000 PCs (more than one load batch of the 512 lifting strands)."""
    rng = np.random.default_rng(77)
    n, n_ctx, R, P, tr, ns = 20000, 8, 7, 5000, 30000, 40000
    rec = random_malformed(rng, n, n_ctx, R, tr)
    from paper_2609_12299_amd import SAMPLE_DTYPE
    smp = np.zeros(ns, SAMPLE_DTYPE)
    smp["ts"] = rng.integers(0, tr + 5, size=ns)
    smp["ctx_key"] = rng.integers(0, n_ctx + 1, size=ns)
    smp["pc"] = rng.integers(0, P, size=ns)
    log(f"[gpu] samples without metrics: n={n} samples={ns} R={R} P={P}")
    g, o = run_both(oracle_mod, rec, R, smp, P)
    assert_samples_parity(g, o, "no metrics")


@pytest.mark.parametrize("cfg,blocks,size,ns,P", [(2, 16, 4096, 1 << 18, 4096),
                                                  (3, 16, 8192, 1 << 19, 20000),
                                                  (5, 0, 1 << 20, 1 << 19, 8192)])
def test_workload_shapes(oracle_mod, tracegen_mod, cfg, blocks, size, ns, P):
    d = tracegen_mod.generate(cfg, blocks=blocks, size=size)
    R = d["num_regions"]
    smp = tracegen_mod.pc_samples(d["records"], ns, P, R, seed=cfg)
    m = np.stack([np.arange(P, dtype=np.float64) % 97, np.ones(P)])
    log(f"[gpu] samples on config {cfg}: records={len(d['records'])} samples={ns} P={P}")
    g, o = run_both(oracle_mod, d["records"], R, smp, P, metrics=m, K=d["num_classes"],
                    cls=d["region_class"], shift=d["group_shift"], G=d["num_groups"])
    assert int(o["counters"][3]) > 0 and int(o["counters"][6]) > 0
    assert_samples_parity(g, o, f"config {cfg}")
