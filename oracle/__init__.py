"""CPU oracle for region attribution over marker traces.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package.  The product library
(``paper_2609_12299_amd``) never imports, links or calls it; the two share no
code.  See ``argus_oracle.cpp`` for the definitions and the paper passages
each step follows.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRCS = [os.path.join(_HERE, f) for f in
         ("argus_oracle.cpp", "argus_oracle_samples.cpp", "argus_oracle_scope.cpp",
          "argus_oracle_probes.cpp", "argus_oracle_handoffs.cpp")]
_LIB = os.path.join(_HERE, "liboracle.so")

NUM_COUNTERS = 32
RS_WIDTH = 142
COUNTER_NAMES = [
    "n_records", "n_valid", "n_bad_kind", "n_bad_region", "n_begin", "n_end",
    "ts_min", "ts_max", "n_ctx", "n_matched", "n_mismatched", "n_unclosed",
    "n_orphan_end", "n_self_nested", "max_level", "n_overlap_skipped",
    "ctx_min", "ctx_max",
]
RS = dict(count=0, incl_sum=1, excl_sum=2, incl_min=3, incl_max=4, excl_min=5,
          excl_max=6, unclosed=7, orphan_end=8, mism_as_begin=9, mism_as_end=10,
          self_nested=11, hist_incl=12, hist_excl=77)

INSTANCE_DTYPE = np.dtype([
    ("t_begin", "<u8"), ("t_end", "<u8"), ("ctx_key", "<u4"), ("parent", "<u4"),
    ("level", "<u4"), ("region_id", "<u2"), ("end_region_id", "<u2"),
])
assert INSTANCE_DTYPE.itemsize == 32


def build(force: bool = True) -> str:
    """Compile the oracle with g++ (single-threaded, -O2)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        # no fused multiply-adds: every product is rounded on its own, as the
        # attribution arithmetic defines
        subprocess.check_call(["g++", "-O2", "-std=c++17", "-Wall", "-ffp-contract=off",
                               "-shared", "-fPIC", *_SRCS, "-o", tmp])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _open(path: str):
    lib = ctypes.CDLL(path)
    f = lib.argus_oracle_run
    f.restype = ctypes.c_int
    f.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint32,
                  ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint32,
                  ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                  ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint64]
    g = lib.argus_oracle_samples
    g.restype = ctypes.c_int
    g.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_void_p, ctypes.c_uint64,
                  ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint32,
                  ctypes.c_void_p] + [ctypes.c_void_p] * 8
    h = lib.argus_oracle_scope
    h.restype = ctypes.c_int
    h.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint32,
                  ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                  ctypes.c_void_p]
    q = lib.argus_oracle_probes
    q.restype = ctypes.c_int
    q.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint32, ctypes.c_void_p,
                  ctypes.c_uint64, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                  ctypes.c_void_p, ctypes.c_uint64, ctypes.c_void_p]
    hh = lib.argus_oracle_handoffs
    hh.restype = ctypes.c_int
    hh.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint32,
                   ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    return lib


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        _lib = _open(_LIB)
    return _lib


class OracleLib:
    """The oracle entry point bound to a specific shared library (tests use
    this to run the pins against deliberately mutated builds)."""

    def __init__(self, path: str):
        self._lib = _open(path)

    def run(self, *args, **kw):
        return run(*args, _lib=self._lib, **kw)

    def samples(self, *args, **kw):
        return samples(*args, _lib=self._lib, **kw)

    def scope(self, *args, **kw):
        return scope(*args, _lib=self._lib, **kw)

    def probes(self, *args, **kw):
        return probes(*args, _lib=self._lib, **kw)

    def handoffs(self, *args, **kw):
        return handoffs(*args, _lib=self._lib, **kw)


def _ptr(a):
    return None if a is None else a.ctypes.data


def run(records: np.ndarray, num_regions: int, num_classes: int = 0, region_class=None,
        group_shift: int = 0, num_groups: int = 0, instances: bool = True, _lib=None) -> dict:
    """Run the oracle on host records (uint8 [N,16] or any 16-byte-itemsize array).

    Returns a dict of numpy arrays: counters [32] u64, region_stats [R,142] u64,
    overlap_group [G,2,K,K] u64 and overlap_global [2,K,K] u64 (K > 0 only),
    instances [n_begin] (INSTANCE_DTYPE) and instance_excl [n_begin] u64.
    """
    rec = np.ascontiguousarray(records)
    nbytes = rec.nbytes
    assert nbytes % 16 == 0, "records are 16 bytes each"
    n = nbytes // 16
    R, K, G = int(num_regions), int(num_classes), int(num_groups)
    cls = None
    if K > 0:
        cls = np.ascontiguousarray(np.asarray(region_class, dtype=np.uint8))
        assert cls.shape == (R,)
    counters = np.zeros(NUM_COUNTERS, np.uint64)
    rstats = np.zeros((R, RS_WIDTH), np.uint64)
    og = np.zeros((G, 2, K, K), np.uint64) if K > 0 else None
    ogl = np.zeros((2, K, K), np.uint64) if K > 0 else None
    if instances:
        # n_begin is at most the number of records.
        kinds = rec.reshape(-1).view(np.uint8).reshape(n, 16)[:, 14] if n else np.zeros(0, np.uint8)
        cap = int(np.count_nonzero(kinds == 1))
        inst = np.zeros(cap, INSTANCE_DTYPE)
        excl = np.zeros(cap, np.uint64)
    else:
        cap, inst, excl = 0, None, None
    lib = _lib if _lib is not None else _load()
    rc = lib.argus_oracle_run(_ptr(rec) if n else None, n, R, K, _ptr(cls), int(group_shift),
                                  G, _ptr(counters), _ptr(rstats), _ptr(og), _ptr(ogl),
                                  _ptr(inst), _ptr(excl), cap)
    if rc != 0:
        raise ValueError(f"argus_oracle_run failed with {rc}")
    out = dict(counters=counters, region_stats=rstats)
    if K > 0:
        out["overlap_group"] = og
        out["overlap_global"] = ogl
    if instances:
        nb = int(counters[4])
        out["instances"] = inst[:nb]
        out["instance_excl"] = excl[:nb]
    return out


def counters_dict(counters: np.ndarray) -> dict:
    return {name: int(counters[i]) for i, name in enumerate(COUNTER_NAMES)}


S_COUNTER_NAMES = ["n_samples", "n_bad_pc", "w_total", "w_attributed", "w_unattributed",
                   "w_inner_unmatched", "n_pairs"]
SAMPLE_DTYPE = np.dtype([("ts", "<u8"), ("ctx_key", "<u4"), ("pc", "<u4")])
assert SAMPLE_DTYPE.itemsize == 16


def samples(instances: np.ndarray, samples_: np.ndarray, num_regions: int, num_pcs: int,
            weights=None, metrics=None, _lib=None) -> dict:
    """PC-sample attribution on host arrays (Section 3.5's alpha, m_hat, H).

    instances: INSTANCE_DTYPE [n] in canonical order; samples_: SAMPLE_DTYPE
    [S] (or any 16-byte-itemsize array); weights: u32 [S] or None (1 each);
    metrics: f64 [M, P] or None.  Returns counters [8] u64, n [P, R] u64,
    alpha [P, R] f64, pc_total [P] u64, pc_owners [P] u32, entropy [P] f64,
    region_total [R] u64 and mhat [M, R] f64.
    """
    inst = np.ascontiguousarray(instances)
    smp = np.ascontiguousarray(samples_)
    assert inst.nbytes % 32 == 0 and smp.nbytes % 16 == 0
    ni, ns = inst.nbytes // 32, smp.nbytes // 16
    R, P = int(num_regions), int(num_pcs)
    w = None if weights is None else np.ascontiguousarray(weights, dtype=np.uint32)
    assert w is None or w.shape == (ns,)
    m = None if metrics is None else np.ascontiguousarray(metrics, dtype=np.float64).reshape(-1, P)
    M = 0 if m is None else m.shape[0]
    out = dict(counters=np.zeros(8, np.uint64), n=np.zeros((P, R), np.uint64),
               alpha=np.zeros((P, R), np.float64), pc_total=np.zeros(P, np.uint64),
               pc_owners=np.zeros(P, np.uint32), entropy=np.zeros(P, np.float64),
               region_total=np.zeros(R, np.uint64), mhat=np.zeros((M, R), np.float64))
    lib = _lib if _lib is not None else _load()
    rc = lib.argus_oracle_samples(_ptr(inst) if ni else None, ni, _ptr(smp) if ns else None, ns,
                                  _ptr(w), R, P, M, _ptr(m) if M else None,
                                  _ptr(out["counters"]), _ptr(out["n"]), _ptr(out["alpha"]),
                                  _ptr(out["pc_total"]), _ptr(out["pc_owners"]),
                                  _ptr(out["entropy"]), _ptr(out["region_total"]),
                                  _ptr(out["mhat"]) if M else None)
    if rc != 0:
        raise ValueError(f"argus_oracle_samples failed with {rc}")
    return out


SC_COUNTER_NAMES = ["n_instances", "n_in_scope", "n_matched", "n_mismatched", "n_unclosed",
                    "n_self_nested", "n_iterations"]
ALL_SCOPE = dict(role_mask=0, role_lo=0, role_hi=0, group_shift=32, group_lo=0, group_hi=0,
                 iter_lo=0, iter_hi=0xFFFFFFFF)


class _Scope(ctypes.Structure):
    _fields_ = [(k, ctypes.c_uint32) for k in ("role_mask", "role_lo", "role_hi", "group_shift",
                                               "group_lo", "group_hi", "iter_lo", "iter_hi")]


def scope(instances: np.ndarray, excl: np.ndarray, num_regions: int, region_mask=None,
          _lib=None, **kw) -> dict:
    """Iteration ordinals and scoped per-region statistics on host arrays.

    Scope fields (keyword arguments) default to "everything": role_mask,
    role_lo, role_hi, group_shift, group_lo, group_hi, iter_lo, iter_hi.
    Returns ordinal [n] u32, stats [R, 142] u64 and counters [8] u64."""
    inst = np.ascontiguousarray(instances)
    ex = np.ascontiguousarray(excl, dtype=np.uint64)
    n = inst.nbytes // 32
    assert ex.shape == (n,)
    f = dict(ALL_SCOPE)
    f.update(kw)
    sc = _Scope(**{k: int(v) for k, v in f.items()})
    R = int(num_regions)
    mask = None if region_mask is None else np.ascontiguousarray(region_mask, dtype=np.uint8)
    out = dict(ordinal=np.zeros(n, np.uint32), stats=np.zeros((R, RS_WIDTH), np.uint64),
               counters=np.zeros(8, np.uint64))
    lib = _lib if _lib is not None else _load()
    rc = lib.argus_oracle_scope(_ptr(inst) if n else None, _ptr(ex) if n else None, n, R,
                                ctypes.byref(sc), _ptr(mask), _ptr(out["ordinal"]),
                                _ptr(out["stats"]), _ptr(out["counters"]))
    if rc != 0:
        raise ValueError(f"argus_oracle_scope failed with {rc}")
    return out


PROBE_DTYPE = np.dtype([("t_start", "<u8"), ("t_end", "<u8"), ("ctx_key", "<u4"),
                        ("iteration", "<u4"), ("op_region", "<u2"), ("pad0", "<u2"),
                        ("pad1", "<u4")])
assert PROBE_DTYPE.itemsize == 32
PG_COLUMNS = ["instance", "count", "sum", "issue", "p0", "p20", "p40", "p60", "p80", "p100"]
PR_COUNTER_NAMES = ["n_probes", "n_bad", "n_joined", "n_unjoined", "n_groups"]


def probes(instances: np.ndarray, num_regions: int, probes_: np.ndarray, _lib=None) -> dict:
    """Join probe intervals (PROBE_DTYPE) to reference instances and
    summarise their latency per joined instance.  Returns ref [n] u32,
    completion [n] u64, groups [G, 10] u64 (columns PG_COLUMNS), mean [G]
    f64 and counters [8] u64."""
    inst = np.ascontiguousarray(instances)
    pr = np.ascontiguousarray(probes_)
    ni, npr = inst.nbytes // 32, pr.nbytes // 32
    cap = max(npr, 1)
    out = dict(ref=np.zeros(npr, np.uint32), completion=np.zeros(npr, np.uint64),
               groups=np.zeros((cap, 10), np.uint64), mean=np.zeros(cap, np.float64),
               counters=np.zeros(8, np.uint64))
    lib = _lib if _lib is not None else _load()
    rc = lib.argus_oracle_probes(_ptr(inst) if ni else None, ni, int(num_regions),
                                 _ptr(pr) if npr else None, npr, _ptr(out["ref"]),
                                 _ptr(out["completion"]), _ptr(out["groups"]), _ptr(out["mean"]),
                                 cap, _ptr(out["counters"]))
    if rc != 0:
        raise ValueError(f"argus_oracle_probes failed with {rc}")
    g = int(out["counters"][4])
    out["groups"] = out["groups"][:g]
    out["mean"] = out["mean"][:g]
    return out


PH_COUNTER_NAMES = ["n_at_level", "n_gaps", "gap_sum"]


def handoffs(instances: np.ndarray, num_regions: int, level: int = 0, _lib=None) -> dict:
    """Gaps between successive level-`level` siblings.  Returns pairs
    [R, R, 4] u64 (count, sum, min, max), hist [65] u64, parent_gap [n] u64
    and counters [8] u64."""
    inst = np.ascontiguousarray(instances)
    n = inst.nbytes // 32
    R = int(num_regions)
    out = dict(pairs=np.zeros((R, R, 4), np.uint64), hist=np.zeros(65, np.uint64),
               parent_gap=np.zeros(n, np.uint64), counters=np.zeros(8, np.uint64))
    lib = _lib if _lib is not None else _load()
    rc = lib.argus_oracle_handoffs(_ptr(inst) if n else None, n, R, int(level), _ptr(out["pairs"]),
                                   _ptr(out["hist"]), _ptr(out["parent_gap"]) if n else None,
                                   _ptr(out["counters"]))
    if rc != 0:
        raise ValueError(f"argus_oracle_handoffs failed with {rc}")
    return out
