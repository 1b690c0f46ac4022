"""Seeded synthetic marker traces (input generation only).

Five workload shapes, after the paper's evaluation (Section 4):

====  ==========================================================  ==========
cfg   shape                                                       records
====  ==========================================================  ==========
1     tiny well-formed: 8 SMs x 4 warps, depth <= 3, 8 regions,  2^16
      shuffled within 4 KiB chunks
2     persistent GEMM (Section 4.1): 256 blocks x 8 warps,        2^24
      producer/consumer stage regions inside per-tile regions
3     decode megakernel (Section 4.2): 256 blocks x 16 warps,    2^26 - 33554
      22 layers x 8 operators + a per-token region, 0.1% of ENDs
      dropped
4     compute/communication overlap (Section 4.3): 256 x 8,       2^25
      flat compute and comm regions on disjoint warps
5     large skewed stress trace: 2048 x 16 warps, Zipf(1.2)       2^28
      records per warp, 1024 regions, depth <= 8, 1% malformed
====  ==========================================================  ==========

This package holds no attribution arithmetic; it is shared by the tests, the
benchmark and the smoke check only as an input source.  Ground-truth instance
lists (configs 1, 2 and 4) are what the generator itself emitted.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "tracegen.c")
_LIB = os.path.join(_HERE, "libtracegen.so")

RECORD_DTYPE = np.dtype([("ts", "<u8"), ("ctx_key", "<u4"), ("region_id", "<u2"),
                         ("kind", "u1"), ("pad", "u1")])
INSTANCE_DTYPE = np.dtype([
    ("t_begin", "<u8"), ("t_end", "<u8"), ("ctx_key", "<u4"), ("parent", "<u4"),
    ("level", "<u4"), ("region_id", "<u2"), ("end_region_id", "<u2"),
])
assert RECORD_DTYPE.itemsize == 16 and INSTANCE_DTYPE.itemsize == 32

DEFAULTS = {1: (8, 4, 2048), 2: (256, 8, 8192), 3: (256, 16, 16384),
            4: (256, 8, 16384), 5: (2048, 16, 1 << 28)}
SEEDS = {1: 0, 2: 1, 3: 2, 4: 3, 5: 4}


def build(force: bool = True) -> str:
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-Wall", "-fopenmp", "-shared",
                               "-fPIC", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        lib = ctypes.CDLL(_LIB)
        lib.tg_size.restype = ctypes.c_int64
        lib.tg_size.argtypes = [ctypes.c_int, ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint64]
        lib.tg_truth_size.restype = ctypes.c_int64
        lib.tg_truth_size.argtypes = lib.tg_size.argtypes
        lib.tg_regions.restype = ctypes.c_int
        lib.tg_regions.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.POINTER(ctypes.c_int)]
        lib.tg_generate.restype = ctypes.c_int64
        lib.tg_generate.argtypes = [ctypes.c_int, ctypes.c_uint64, ctypes.c_uint32,
                                    ctypes.c_uint32, ctypes.c_uint64, ctypes.c_void_p,
                                    ctypes.c_uint64, ctypes.c_void_p, ctypes.c_uint64,
                                    ctypes.c_int]
        _lib = lib
    return _lib


def _log2(v: int) -> int:
    assert v > 0 and v & (v - 1) == 0, "warps per block must be a power of two"
    return v.bit_length() - 1


def generate(cfg: int, seed: int | None = None, blocks: int = 0, warps: int = 0,
             size: int = 0, truth: bool = False, threads: int = 0, out=None) -> dict:
    """Generate configuration `cfg` (1..5).

    blocks / warps / size default to the full configuration when 0; `size`
    is records per warp for configs 1-4 and the total record count for 5.
    `out` may be a preallocated uint8 buffer (e.g. pinned) of at least
    16 * N bytes.  Returns a dict with the records (uint8 [N, 16]) and the
    attribution parameters of the shape (num_regions, num_classes,
    region_class, group_shift, num_groups), plus `truth` for configs
    1, 2 and 4 when asked.
    """
    lib = _load()
    if seed is None:
        seed = SEEDS[cfg]
    b0, w0, _ = DEFAULTS[cfg]
    B = blocks or b0
    W = warps or w0
    n = lib.tg_size(cfg, B, W, size)
    if n < 0:
        raise ValueError("bad configuration")
    if out is None:
        rec = np.empty((n, 16), np.uint8)
    else:
        rec = out.reshape(-1)[: n * 16].reshape(n, 16)
    tn = lib.tg_truth_size(cfg, B, W, size) if truth else 0
    tr = np.empty(tn, INSTANCE_DTYPE) if tn > 0 else None
    got = lib.tg_generate(cfg, seed, B, W, size, rec.ctypes.data, n,
                          tr.ctypes.data if tr is not None else None, tn, threads)
    if got != n:
        raise RuntimeError(f"tg_generate returned {got}, expected {n}")
    cls = np.zeros(65536, np.uint8)
    k = ctypes.c_int(0)
    R = lib.tg_regions(cfg, cls.ctypes.data, ctypes.byref(k))
    out_d = dict(records=rec, num_regions=R, num_classes=k.value,
                 region_class=cls[:R].copy(), group_shift=_log2(W), num_groups=B,
                 cfg=cfg, seed=seed, blocks=B, warps=W)
    if tr is not None:
        out_d["truth"] = tr
    return out_d


def as_records(rec_u8: np.ndarray) -> np.ndarray:
    """View uint8 [N,16] records as the structured record dtype."""
    return rec_u8.reshape(-1).view(RECORD_DTYPE)


def make_records(rows) -> np.ndarray:
    """Build uint8 [N,16] records from (ts, ctx, region, kind) tuples."""
    a = np.zeros(len(rows), RECORD_DTYPE)
    for i, (ts, ctx, region, kind) in enumerate(rows):
        a[i] = (ts, ctx, region, kind, 0)
    return a.view(np.uint8).reshape(len(rows), 16)


SAMPLE_DTYPE = np.dtype([("ts", "<u8"), ("ctx_key", "<u4"), ("pc", "<u4")])


def pc_samples(records: np.ndarray, n_samples: int, num_pcs: int, num_regions: int,
               seed: int = 0, shared_pcs: int = 64, p_shared: float = 0.2,
               max_offset: int = 400) -> np.ndarray:
    """Synthetic PC samples shaped like a sampling run over the same kernel.

    Each sample copies the context and the time (plus U[0, max_offset)) of
    a random marker record, so samples follow the trace's layout and fall
    inside, between and after regions.  Its PC is drawn from a block of PCs
    tied to that marker's region id (the code of the region), or, with
    probability p_shared, from `shared_pcs` helper PCs used by every region
    (the shared helpers and epilogues that make ownership ambiguous).  About
    1 in 1000 samples gets pc = num_pcs (out of range).  No attribution is
    computed here.  Returns SAMPLE_DTYPE [n_samples] in the records' order.
    """
    rng = np.random.default_rng(seed)
    rec = as_records(records)
    n = len(rec)
    idx = np.sort(rng.integers(0, n, size=n_samples)) if n else np.zeros(0, np.int64)
    out = np.zeros(n_samples, SAMPLE_DTYPE)
    if n == 0:
        return out
    out["ts"] = rec["ts"][idx] + rng.integers(0, max_offset, size=n_samples).astype(np.uint64)
    out["ctx_key"] = rec["ctx_key"][idx]
    block = max(1, (num_pcs - shared_pcs) // max(1, num_regions))
    reg = rec["region_id"][idx].astype(np.int64) % max(1, num_regions)
    own = shared_pcs + reg * block + rng.integers(0, block, size=n_samples)
    shared = rng.random(n_samples) < p_shared
    pc = np.where(shared, rng.integers(0, shared_pcs, size=n_samples), own)
    pc = np.minimum(pc, num_pcs - 1)
    pc[rng.random(n_samples) < 0.001] = num_pcs
    out["pc"] = pc.astype(np.uint32)
    return out


PROBE_DTYPE = np.dtype([("t_start", "<u8"), ("t_end", "<u8"), ("ctx_key", "<u4"),
                        ("iteration", "<u4"), ("op_region", "<u2"), ("pad0", "<u2"),
                        ("pad1", "<u4")])


def probes_for(ops, n_ctx: int, iterations: int, repeats: int, seed: int = 0,
               mu: float = 6.5, sigma: float = 0.7, p_missing: float = 0.01) -> np.ndarray:
    """Synthetic forced-completion probe intervals: for every context in
    [0, n_ctx), operation region in `ops` and iteration in [0, iterations),
    `repeats` probe runs each measure one interval whose length is
    LogNormal(mu, sigma) cycles, on a clock of their own (start times
    unrelated to the reference trace).  A fraction p_missing asks for an
    iteration beyond `iterations` (nothing to join).  No join is computed
    here.  Returns PROBE_DTYPE records in (repeat, context, op, iteration)
    order."""
    rng = np.random.default_rng(seed)
    ops = np.asarray(ops, np.uint16)
    c, o, i = np.meshgrid(np.arange(n_ctx), np.arange(len(ops)), np.arange(iterations),
                          indexing="ij")
    base = np.stack([c.ravel(), o.ravel(), i.ravel()], axis=1)
    n = len(base) * repeats
    out = np.zeros(n, PROBE_DTYPE)
    rows = np.tile(base, (repeats, 1))
    out["ctx_key"] = rows[:, 0]
    out["op_region"] = ops[rows[:, 1]]
    it = rows[:, 2].astype(np.uint32)
    miss = rng.random(n) < p_missing
    it[miss] += np.uint32(iterations)
    out["iteration"] = it
    out["t_start"] = rng.integers(0, 1 << 40, size=n).astype(np.uint64)
    lat = np.maximum(1, np.round(rng.lognormal(mu, sigma, size=n))).astype(np.uint64)
    out["t_end"] = out["t_start"] + lat
    return out
