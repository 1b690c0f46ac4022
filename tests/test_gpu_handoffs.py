"""Phase-handoff gaps on the GPU (argus_attr_handoffs) against the oracle,
on the instance array argus_attr_run wrote on the device.  All integers:
identical."""
from __future__ import annotations

import numpy as np
import pytest

from golden_util import random_malformed, records_from_rows
from gpu_util import log

pytestmark = pytest.mark.gpu


def run_both(oracle_mod, rec_u8, R, levels, K=0, cls=None, shift=0, G=0):
    import torch

    from paper_2609_12299_amd import RegionAttribution, phase_handoffs
    n = rec_u8.shape[0]
    ra = RegionAttribution(R, K, cls, shift, G, max_records=max(n, 1))
    rec = torch.from_numpy(np.ascontiguousarray(rec_u8).reshape(-1)).to("cuda")
    out = ra.run(rec)
    oi = oracle_mod.run(rec_u8, R, K, cls, shift, G)["instances"]
    res = []
    for L in levels:
        g = phase_handoffs(out["instances"], out["counters"][4:5], R, level=L)
        torch.cuda.synchronize()
        g = {k: v.cpu().numpy() for k, v in g.items() if not k.startswith("_")}
        res.append((L, g, oracle_mod.handoffs(oi, R, L)))
    ra.close()
    return res


def assert_parity(g, o, what):
    nb = len(o["parent_gap"])
    for k in ("pairs", "hist", "counters"):
        np.testing.assert_array_equal(g[k], o[k], err_msg=f"{what}: {k}")
    np.testing.assert_array_equal(g["parent_gap"][:nb], o["parent_gap"], err_msg=f"{what}: parent_gap")


def test_hand_steps(oracle_mod):
    B, E = 1, 2
    rows = [(0, 0, 0, B), (10, 0, 1, B), (20, 0, 1, E), (25, 0, 2, B), (40, 0, 2, E),
            (60, 0, 3, B), (70, 0, 3, E), (100, 0, 0, E),
            (100, 0, 0, B), (110, 0, 1, B), (120, 0, 1, E), (121, 0, 2, B), (190, 0, 2, E),
            (200, 0, 0, E)]
    for L, g, o in run_both(oracle_mod, records_from_rows(rows), 4, [0, 1, 2]):
        assert_parity(g, o, f"hand L={L}")
    assert g is not None


@pytest.mark.parametrize("n,n_ctx,R,tr", [(0, 2, 2, 10), (3, 1, 2, 10), (4097, 5, 7, 3000),
                                          (30001, 17, 40, 40000), (100000, 64, 300, 1 << 20),
                                          # millions of distinct region pairs: every block's LDS
                                          # table fills and pairs go to the output rows directly,
                                          # and the keys homed in one merge range across all the
                                          # tables outnumber the merge table's slots
                                          (8000000, 16, 3000, 1 << 22)])
def test_random(oracle_mod, n, n_ctx, R, tr):
    rng = np.random.default_rng(n + R + 5)
    rec = random_malformed(rng, n, n_ctx, R, tr)
    log(f"[gpu] handoffs random: n={n} R={R}")
    for L, g, o in run_both(oracle_mod, rec, R, [0, 1, 3]):
        assert_parity(g, o, f"random n={n} L={L}")


def test_decode_megakernel_steps(oracle_mod, tracegen_mod):
    """Operator phases (level 1) inside each token step of the decode-
    megakernel-shaped trace: per-step handoff totals and operator pairs."""
    d = tracegen_mod.generate(3, blocks=8, size=16384)
    log(f"[gpu] handoffs on config 3: records={len(d['records'])}")
    for L, g, o in run_both(oracle_mod, d["records"], d["num_regions"], [0, 1], K=d["num_classes"],
                            cls=d["region_class"], shift=d["group_shift"], G=d["num_groups"]):
        assert int(o["counters"][1]) > 0
        assert_parity(g, o, f"config 3 L={L}")
