"""argus_attr_run under HIP graph capture: the whole run (output
initialisation by fill kernels, no memset nodes, device-planned passes) is
captured once into a torch.cuda.CUDAGraph and replayed several times, with
eager work of the program and synchronisations between the replays.  Every
replay must reproduce the oracle bit for bit."""
from __future__ import annotations

import numpy as np
import pytest

from gpu_util import assert_parity, log, oracle_run

pytestmark = pytest.mark.gpu


def _params(d):
    return {k: d[k] for k in ("num_regions", "num_classes", "region_class", "group_shift", "num_groups")}


@pytest.mark.parametrize("cfg,blocks,size", [(1, 0, 0), (3, 8, 4096)])
def test_run_captured_in_graph(oracle_mod, tracegen_mod, cfg, blocks, size):
    import torch

    from paper_2609_12299_amd import RegionAttribution, to_host
    d = tracegen_mod.generate(cfg, blocks=blocks, size=size)
    p = _params(d)
    n = len(d["records"])
    log(f"[gpu] graph capture: config {cfg}, n={n}")
    o = oracle_run(oracle_mod, d["records"], p)
    ra = RegionAttribution(p["num_regions"], p["num_classes"], p["region_class"], p["group_shift"],
                           p["num_groups"], max_records=n)
    rec = torch.from_numpy(d["records"].reshape(-1)).to("cuda")
    out = ra.alloc(n)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):  # warm-up outside capture: workspace allocated, device checked
        ra.run(rec, out, stream=s)
    s.synchronize()
    assert_parity(to_host(out), o, what=f"graph cfg{cfg} eager")
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        ra.run(rec, out)
    torch.cuda.synchronize()
    scratch = torch.empty(1 << 20, dtype=torch.int64, device="cuda")
    for rep in range(3):
        for v in out.values():  # poison the outputs: the replay must rewrite all of them
            v.fill_(0x5A)
        scratch.random_()  # unrelated eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert_parity(to_host(out), o, what=f"graph cfg{cfg} replay {rep}")
    del g
    ra.close()
