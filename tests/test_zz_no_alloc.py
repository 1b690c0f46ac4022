"""argus_attr_run_noalloc, the entry point without a workspace argument (its
workspace is the library's built-in per-device array), against
argus_attr_run with a caller workspace: two calls in a row on one handle, the
second with a smaller input, each compared output by output, bit for bit.
The built-in array keeps the first call's contents, so the second call also
checks that every call initialises what it reads."""
from __future__ import annotations

import numpy as np
import pytest

from gpu_util import assert_parity, log

pytestmark = pytest.mark.gpu


def _malformed(rng, n, n_ctx, R):
    """Random marker records: mixed kinds (some invalid), regions (some out
    of range), contexts and timestamps with ties."""
    from golden_util import RECORD_DTYPE
    rec = np.zeros(n, RECORD_DTYPE)
    rec["ts"] = rng.integers(0, 1 << 20, size=n, dtype=np.uint64)
    rec["ctx_key"] = rng.integers(0, n_ctx, size=n, dtype=np.uint32)
    rec["region_id"] = rng.integers(0, R + 1, size=n)
    rec["kind"] = rng.choice(np.array([1, 2, 0], np.uint8), size=n, p=[0.49, 0.49, 0.02])
    return rec.view(np.uint8).reshape(n, 16)


def _both(ra, rec_u8, stream):
    import torch

    from paper_2609_12299_amd import to_host
    n = rec_u8.shape[0]
    rec = torch.from_numpy(np.ascontiguousarray(rec_u8).reshape(-1)).to("cuda")
    ref_out = ra.alloc(n)
    ra.run(rec, ref_out, stream=stream)
    stream.synchronize()
    ref = to_host(ref_out)
    # outputs poisoned first: the entry point must initialise every one of them
    out = ra.alloc(n)
    for v in out.values():
        v.fill_(0xA5)
    ra.run_noalloc(rec, out, stream=stream)
    stream.synchronize()
    return to_host(out), ref


def test_noalloc_matches_run_two_calls(tracegen_mod):
    import torch

    from paper_2609_12299_amd import NOALLOC_SCRATCH_BYTES, ArgusError, RegionAttribution
    d = tracegen_mod.generate(1)  # 2^16 records, 32 contexts, 2 classes over 8 groups
    R, K, G, shift = d["num_regions"], d["num_classes"], d["num_groups"], d["group_shift"]
    n1 = len(d["records"])
    ra = RegionAttribution(R, K, d["region_class"], shift, G, max_records=1 << 20)
    assert ra.workspace(n1)[1] <= NOALLOC_SCRATCH_BYTES
    stream = torch.cuda.Stream()
    log(f"[gpu] noalloc call 1: n={n1}")
    g, ref = _both(ra, d["records"], stream)
    assert int(ref["counters"][9]) > 0
    assert_parity(g, ref, what="noalloc call 1")
    rng = np.random.default_rng(7)
    rec2 = _malformed(rng, 5001, 12, R)
    log("[gpu] noalloc call 2: n=5001")
    g, ref = _both(ra, rec2, stream)
    assert_parity(g, ref, what="noalloc call 2")
    # beyond the built-in workspace: a clear error before any GPU work
    big = 1 << 20
    assert ra.workspace(big)[1] > NOALLOC_SCRATCH_BYTES
    big_rec = torch.zeros(big * 16, dtype=torch.uint8, device="cuda")
    with pytest.raises(ArgusError, match="built-in workspace"):
        ra.run_noalloc(big_rec, ra.alloc(1))
    ra.close()
