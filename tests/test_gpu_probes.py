"""Probe <-> reference join on the GPU (argus_attr_probes) against the
oracle.  The reference instances come from argus_attr_run on the device
(count read on the device); the oracle joins against its own.  Every output
is an integer except the mean, which is one correctly rounded division of
two integers: all must be identical."""
from __future__ import annotations

import numpy as np
import pytest

from golden_util import random_malformed, records_from_rows
from gpu_util import log

pytestmark = pytest.mark.gpu


def run_both(oracle_mod, rec_u8, R, probes, K=0, cls=None, shift=0, G=0):
    import torch

    from paper_2609_12299_amd import RegionAttribution, join_probes
    n = rec_u8.shape[0]
    ra = RegionAttribution(R, K, cls, shift, G, max_records=max(n, 1))
    rec = torch.from_numpy(np.ascontiguousarray(rec_u8).reshape(-1)).to("cuda")
    out = ra.run(rec)
    pt = torch.from_numpy(np.ascontiguousarray(probes).view(np.uint8).reshape(-1)).to("cuda")
    g = join_probes(out["instances"], out["counters"][4:5], pt, R)
    torch.cuda.synchronize()
    g = {k: v.cpu().numpy() for k, v in g.items() if not k.startswith("_")}
    ra.close()
    oi = oracle_mod.run(rec_u8, R, K, cls, shift, G)["instances"]
    return g, oracle_mod.probes(oi, R, probes)


def assert_probe_parity(g, o, what):
    npr = len(o["ref"])
    np.testing.assert_array_equal(g["counters"], o["counters"], err_msg=f"{what}: counters")
    np.testing.assert_array_equal(g["ref"][:npr], o["ref"], err_msg=f"{what}: ref")
    np.testing.assert_array_equal(g["completion"][:npr], o["completion"], err_msg=f"{what}: completion")
    ng = int(o["counters"][4])
    np.testing.assert_array_equal(g["groups"][:ng], o["groups"], err_msg=f"{what}: groups")
    assert g["mean"][:ng].tobytes() == o["mean"].tobytes(), f"{what}: mean"


def _probes(rng, m, n_ctx, R, iters):
    from paper_2609_12299_amd import PROBE_DTYPE
    pr = np.zeros(m, PROBE_DTYPE)
    pr["t_start"] = rng.integers(0, 1 << 40, size=m)
    pr["t_end"] = pr["t_start"] + rng.integers(0, 5000, size=m).astype(np.uint64)
    bad = rng.random(m) < 0.01
    pr["t_end"][bad] = pr["t_start"][bad] - np.uint64(1)
    pr["ctx_key"] = rng.integers(0, n_ctx + 1, size=m)
    pr["iteration"] = rng.integers(0, iters, size=m)
    pr["op_region"] = rng.integers(0, R + 1, size=m)
    return pr


def test_hand(oracle_mod):
    B, E = 1, 2
    rows = []
    for t in (100, 200, 300):
        rows += [(t - 5, 0, 0, B), (t, 0, 1, B), (t + 50, 0, 1, E), (t + 60, 0, 0, E)]
    from paper_2609_12299_amd import PROBE_DTYPE
    pr = np.zeros(6, PROBE_DTYPE)
    for i, d in enumerate((30, 10, 50, 20, 40)):
        pr[i] = (10 ** 9, 10 ** 9 + d, 0, 1, 1, 0, 0)
    pr[5] = (0, 5, 0, 9, 1, 0, 0)  # iteration 9: nothing to join
    g, o = run_both(oracle_mod, records_from_rows(rows), 2, pr)
    assert g["groups"][0].tolist() == [3, 5, 150, 200, 10, 10, 20, 30, 40, 50]
    assert_probe_parity(g, o, "hand")


@pytest.mark.parametrize("n,m,n_ctx,R,iters", [(0, 10, 2, 2, 3), (50, 0, 2, 2, 3),
                                               (4097, 5000, 5, 7, 40), (30001, 4097, 17, 300, 30),
                                               (100000, 100000, 64, 9, 200)])
def test_random(oracle_mod, n, m, n_ctx, R, iters):
    rng = np.random.default_rng(n + m)
    rec = random_malformed(rng, n, n_ctx, R, max(n, 10))
    log(f"[gpu] probes random: n={n} probes={m} R={R}")
    g, o = run_both(oracle_mod, rec, R, _probes(rng, m, n_ctx, R, iters))
    assert_probe_parity(g, o, f"random n={n} m={m}")


def test_persistent_gemm_probes(oracle_mod, tracegen_mod):
    """Probes of the producer's load regions (1, 2: load_A, load_B) and the
    consumer's mma region (7) over sixteen iterations, five repeats each, on
    the persistent-GEMM-shaped reference."""
    d = tracegen_mod.generate(2, blocks=32, size=4096)
    pr = tracegen_mod.probes_for([1, 2, 7], 32 * 8, 16, 5, seed=9)
    log(f"[gpu] probes on config 2: records={len(d['records'])} probes={len(pr)}")
    g, o = run_both(oracle_mod, d["records"], d["num_regions"], pr, K=d["num_classes"],
                    cls=d["region_class"], shift=d["group_shift"], G=d["num_groups"])
    assert int(o["counters"][2]) > 0 and int(o["counters"][4]) > 0
    assert_probe_parity(g, o, "config 2")


@pytest.mark.parametrize("spread", ["full", "equal", "byte5"])
def test_latency_spreads(oracle_mod, spread):
    """The (instance, latency) sort skips the passes whose byte is the same
    for every probe: latencies varying in all eight bytes (no pass skipped),
    all zero (every latency pass skipped), and varying only in bytes 0 and 5
    (the passes between and after them skipped)."""
    rng = np.random.default_rng({"full": 1, "equal": 2, "byte5": 3}[spread])
    rec = random_malformed(rng, 30001, 17, 9, 40000)
    pr = _probes(rng, 20000, 17, 9, 30)
    ok = pr["t_end"] >= pr["t_start"]
    if spread == "full":
        lat = rng.integers(0, 1 << 62, size=len(pr), dtype=np.uint64)
        pr["t_start"] = rng.integers(0, 1 << 62, size=len(pr), dtype=np.uint64)
    elif spread == "equal":
        # 0, as unjoined and malformed probes have: every latency byte is constant
        lat = np.zeros(len(pr), np.uint64)
    else:
        lat = (rng.integers(0, 256, size=len(pr)).astype(np.uint64) << np.uint64(40)) | np.uint64(3)
    pr["t_end"] = np.where(ok, pr["t_start"] + lat, pr["t_start"] - np.uint64(1))
    log(f"[gpu] probes latency spread {spread}")
    g, o = run_both(oracle_mod, rec, 9, pr)
    assert int(o["counters"][2]) > 0
    assert_probe_parity(g, o, f"spread {spread}")
