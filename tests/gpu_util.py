"""Helpers for the GPU parity tests: run the HIP library through its C ABI
(the torch wrapper only marshals arguments) and compare with the oracle."""
from __future__ import annotations

import sys

import numpy as np


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def gpu_run(rec_u8: np.ndarray, p: dict, force_full: bool = False, instances: bool = True,
            stream=None, repeat: int = 1, force_event: bool = False, with_plan: bool = False,
            force_radix: bool = False) -> dict:
    import torch

    from paper_2609_12299_amd import RegionAttribution, to_host
    n = rec_u8.shape[0]
    ra = RegionAttribution(p["num_regions"], p.get("num_classes", 0), p.get("region_class"),
                           p.get("group_shift", 0), p.get("num_groups", 0),
                           max_records=max(n, 1), instances=instances, instance_excl=instances,
                           force_full_sort=force_full, force_event_sort=force_event,
                           force_record_radix=force_radix)
    rec = torch.from_numpy(np.ascontiguousarray(rec_u8).reshape(-1)).to("cuda")
    outs = []
    for _ in range(repeat):
        if stream is not None:
            with torch.cuda.stream(stream):
                out = ra.run(rec, stream=stream)
            stream.synchronize()
        else:
            out = ra.run(rec)
            torch.cuda.synchronize()
        res = to_host(out)
        if with_plan and n > 0:
            res["_plan"] = ra.plan()
        outs.append(res)
    ra.close()
    return outs[0] if repeat == 1 else outs


def oracle_run(oracle_mod, rec_u8: np.ndarray, p: dict, instances: bool = True) -> dict:
    return oracle_mod.run(rec_u8, p["num_regions"], p.get("num_classes", 0), p.get("region_class"),
                          p.get("group_shift", 0), p.get("num_groups", 0), instances=instances)


def assert_parity(g: dict, o: dict, instances: bool = True, what: str = "") -> None:
    """Bit-exact comparison of every output (all integers)."""
    assert int(g["counters"][31]) == 0, f"{what}: internal error flag {int(g['counters'][31])}"
    np.testing.assert_array_equal(g["counters"], o["counters"], err_msg=f"{what}: counters")
    np.testing.assert_array_equal(g["region_stats"], o["region_stats"], err_msg=f"{what}: region_stats")
    if "overlap_group" in o:
        np.testing.assert_array_equal(g["overlap_group"], o["overlap_group"], err_msg=f"{what}: overlap_group")
        np.testing.assert_array_equal(g["overlap_global"], o["overlap_global"], err_msg=f"{what}: overlap_global")
    if instances:
        gi, oi = g["instances"], o["instances"]
        assert gi.shape == oi.shape, f"{what}: {gi.shape} instances vs {oi.shape}"
        if gi.tobytes() != oi.tobytes():
            diff = np.nonzero((gi.view(np.uint8).reshape(-1, 32) != oi.view(np.uint8).reshape(-1, 32)).any(axis=1))[0]
            k = diff[0]
            raise AssertionError(f"{what}: {len(diff)} instances differ; first {k}: gpu {gi[k]} oracle {oi[k]}")
        np.testing.assert_array_equal(g["instance_excl"], o["instance_excl"], err_msg=f"{what}: excl")
