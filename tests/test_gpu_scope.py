"""Iteration ordinals and scoped statistics on the GPU (argus_attr_scope)
against the oracle.  The GPU side works on the instance array and exclusive
times that argus_attr_run wrote on the device (instance count read on the
device); the oracle side on the oracle's own.  All outputs are integers and
must be identical."""
from __future__ import annotations

import numpy as np
import pytest

from golden_util import random_malformed
from gpu_util import log

pytestmark = pytest.mark.gpu


def run_both(oracle_mod, rec_u8, R, scopes, masks=None, K=0, cls=None, shift=0, G=0):
    import torch

    from paper_2609_12299_amd import RegionAttribution, scope_statistics
    n = rec_u8.shape[0]
    ra = RegionAttribution(R, K, cls, shift, G, max_records=max(n, 1))
    rec = torch.from_numpy(np.ascontiguousarray(rec_u8).reshape(-1)).to("cuda")
    out = ra.run(rec)
    o = oracle_mod.run(rec_u8, R, K, cls, shift, G)
    nb = int(o["counters"][4])
    res = []
    for i, sc in enumerate(scopes):
        mask = None if masks is None else masks[i]
        tm = torch.from_numpy(mask).to("cuda") if mask is not None else None
        g = scope_statistics(out["instances"], out["instance_excl"], out["counters"][4:5], R,
                             region_mask=tm, **sc)
        torch.cuda.synchronize()
        g = {k: v.cpu().numpy() for k, v in g.items() if not k.startswith("_")}
        w = oracle_mod.scope(o["instances"], o["instance_excl"], R, region_mask=mask, **sc)
        res.append((g, w, nb))
    ra.close()
    return res


def assert_scope_parity(g, w, nb, what):
    np.testing.assert_array_equal(g["ordinal"][:nb], w["ordinal"], err_msg=f"{what}: ordinal")
    np.testing.assert_array_equal(g["counters"], w["counters"], err_msg=f"{what}: counters")
    np.testing.assert_array_equal(g["stats"], w["stats"], err_msg=f"{what}: stats")


SCOPES = [dict(), dict(iter_lo=1, iter_hi=3), dict(role_mask=3, role_lo=1, role_hi=2),
          dict(group_shift=2, group_lo=1, group_hi=5), dict(iter_lo=0, iter_hi=0, role_mask=1,
                                                              role_lo=0, role_hi=0)]


@pytest.mark.parametrize("n,n_ctx,R,tr", [(0, 3, 3, 10), (1, 1, 2, 5), (4095, 5, 7, 3000),
                                          (4097, 9, 300, 4000), (8193, 3, 2, 100),
                                          (30001, 17, 9, 40000), (100000, 64, 700, 1 << 20),
                                          # 4096 regions: the chunk walk's widest case (a
                                          # ballot per region bit, 12 of them, and 64 KiB of
                                          # counters per block)
                                          (60000, 11, 4096, 80000),
                                          # more than 4096 regions: the whole-array sort path
                                          (20000, 7, 5000, 30000),
                                          # three contexts over ~370 chunks of 4096 instances:
                                          # carries through whole chunks and across segments
                                          # of 256 chunks
                                          (3000000, 3, 40, 1 << 22)])
def test_random_malformed(oracle_mod, n, n_ctx, R, tr):
    rng = np.random.default_rng(n + R)
    rec = random_malformed(rng, n, n_ctx, R, tr)
    masks = [None] * (len(SCOPES) - 1) + [(rng.random(R) < 0.5).astype(np.uint8)]
    log(f"[gpu] scope random: n={n} R={R}")
    for i, (g, w, nb) in enumerate(run_both(oracle_mod, rec, R, SCOPES, masks)):
        assert_scope_parity(g, w, nb, f"random n={n} scope {i}")


@pytest.mark.parametrize("cfg,blocks,size,scopes", [
    # producer warps (0, 1 of 8) of the persistent GEMM, and consumer warps
    (2, 32, 4096, [dict(role_mask=7, role_lo=0, role_hi=1), dict(role_mask=7, role_lo=2, role_hi=7)]),
    # sixteen token iterations of the decode megakernel, and one SM subset
    (3, 16, 16384, [dict(iter_lo=0, iter_hi=15), dict(group_shift=4, group_lo=3, group_hi=7)]),
    (5, 0, 1 << 20, [dict(), dict(iter_lo=2, iter_hi=9)]),
])
def test_workload_shapes(oracle_mod, tracegen_mod, cfg, blocks, size, scopes):
    d = tracegen_mod.generate(cfg, blocks=blocks, size=size)
    log(f"[gpu] scope on config {cfg}: records={len(d['records'])}")
    for i, (g, w, nb) in enumerate(run_both(oracle_mod, d["records"], d["num_regions"], scopes,
                                            K=d["num_classes"], cls=d["region_class"],
                                            shift=d["group_shift"], G=d["num_groups"])):
        assert int(w["counters"][1]) > 0
        assert_scope_parity(g, w, nb, f"config {cfg} scope {i}")
