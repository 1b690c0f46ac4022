"""The steps that work on the instances of a run, at the sizes and shapes
bench.py times them (--part samples / scope / probes / handoffs), compared
whole with the oracle: PC-sample attribution on the 2^26-record decode-
megakernel trace with 2^24 samples over 65536 PCs; iteration ordinals and
scoped statistics on the 2^28-record trace; the probe join on the 2^24-
record persistent-GEMM trace; phase handoffs of the operator phases of the
decode megakernel."""
from __future__ import annotations

import numpy as np
import pytest

from gpu_util import log
from test_gpu_handoffs import assert_parity as assert_handoff_parity
from test_gpu_probes import assert_probe_parity
from test_gpu_samples import assert_samples_parity
from test_gpu_scope import assert_scope_parity

pytestmark = pytest.mark.gpu


def _device_run(d):
    import torch

    from paper_2609_12299_amd import RegionAttribution
    rec_np = d["records"]
    ra = RegionAttribution(d["num_regions"], d["num_classes"], d["region_class"], d["group_shift"],
                           d["num_groups"], max_records=len(rec_np))
    out = ra.run(torch.from_numpy(rec_np.reshape(-1)).to("cuda"))
    torch.cuda.synchronize()
    return ra, out


def _oracle_instances(oracle_mod, d):
    o = oracle_mod.run(d["records"], d["num_regions"], d["num_classes"], d["region_class"],
                       d["group_shift"], d["num_groups"])
    return o["instances"], o["instance_excl"]


@pytest.mark.timeout(900)
def test_samples_decode_megakernel(oracle_mod, tracegen_mod):
    import torch

    from paper_2609_12299_amd import attribute_samples
    d = tracegen_mod.generate(3, threads=16)
    R, S, P = d["num_regions"], 1 << 24, 65536
    smp = tracegen_mod.pc_samples(d["records"], S, P, R, seed=1)
    met = np.stack([np.arange(P, dtype=np.float64) % 97, np.ones(P)])
    log(f"[gpu] full-size samples: records={len(d['records'])} samples={S} P={P}")
    ra, out = _device_run(d)
    g = attribute_samples(out["instances"], out["counters"][4:5],
                          torch.from_numpy(smp.view(np.uint8).reshape(-1)).to("cuda"), R, P,
                          metrics=torch.from_numpy(met).to("cuda"))
    torch.cuda.synchronize()
    g = {k: v.cpu().numpy() for k, v in g.items()}
    ra.close()
    del out
    oi, _ = _oracle_instances(oracle_mod, d)
    log("[gpu] full-size samples: oracle")
    o = oracle_mod.samples(oi, smp, R, P, metrics=met)
    assert_samples_parity(g, o, "full-size samples")


@pytest.mark.timeout(900)
def test_handoffs_decode_megakernel(oracle_mod, tracegen_mod):
    import torch

    from paper_2609_12299_amd import phase_handoffs
    d = tracegen_mod.generate(3, threads=16)
    R = d["num_regions"]
    ra, out = _device_run(d)
    log(f"[gpu] full-size handoffs: records={len(d['records'])}")
    res = {}
    for L in (0, 1):
        g = phase_handoffs(out["instances"], out["counters"][4:5], R, level=L)
        torch.cuda.synchronize()
        res[L] = {k: v.cpu().numpy() for k, v in g.items() if not k.startswith("_")}
    ra.close()
    del out
    oi, _ = _oracle_instances(oracle_mod, d)
    for L in (0, 1):
        o = oracle_mod.handoffs(oi, R, L)
        assert int(o["counters"][1]) > 0
        assert_handoff_parity(res[L], o, f"full-size handoffs L={L}")


@pytest.mark.timeout(900)
def test_probes_persistent_gemm(oracle_mod, tracegen_mod):
    import torch

    from paper_2609_12299_amd import join_probes
    d = tracegen_mod.generate(2, threads=16)
    R = d["num_regions"]
    pr = tracegen_mod.probes_for([1, 2, 7], d["blocks"] * d["warps"], 16, 5, seed=9)
    ra, out = _device_run(d)
    log(f"[gpu] full-size probes: records={len(d['records'])} probes={len(pr)}")
    g = join_probes(out["instances"], out["counters"][4:5],
                    torch.from_numpy(pr.view(np.uint8).reshape(-1)).to("cuda"), R)
    torch.cuda.synchronize()
    g = {k: v.cpu().numpy() for k, v in g.items() if not k.startswith("_")}
    ra.close()
    del out
    oi, _ = _oracle_instances(oracle_mod, d)
    o = oracle_mod.probes(oi, R, pr)
    assert int(o["counters"][4]) > 0
    assert_probe_parity(g, o, "full-size probes")


@pytest.mark.timeout(1200)
def test_scope_large_trace(oracle_mod, tracegen_mod):
    import torch

    from paper_2609_12299_amd import scope_statistics
    d = tracegen_mod.generate(5, threads=16)
    R = d["num_regions"]
    ra, out = _device_run(d)
    log(f"[gpu] full-size scope: records={len(d['records'])}")
    g = scope_statistics(out["instances"], out["instance_excl"], out["counters"][4:5], R,
                         iter_lo=0, iter_hi=15)
    torch.cuda.synchronize()
    nb = int(out["counters"][4].item())
    g = {k: v.cpu().numpy() for k, v in g.items() if not k.startswith("_")}
    ra.close()
    del out
    oi, oe = _oracle_instances(oracle_mod, d)
    log("[gpu] full-size scope: oracle")
    w = oracle_mod.scope(oi, oe, R, iter_lo=0, iter_hi=15)
    assert_scope_parity(g, w, nb, "full-size scope")
