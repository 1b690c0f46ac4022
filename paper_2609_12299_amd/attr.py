"""Python binding of the region-attribution C ABI (include/argus_attr.h).

The functions named ``argus_attr_*`` are one-to-one wrappers (argument
marshalling only).  :class:`RegionAttribution` adds what a PyTorch caller
needs: it allocates outputs and the workspace as torch tensors on the current
device and runs on the current torch stream.  Every step of the computation
runs in the HIP kernels of libargus_attr.so; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libargus_attr.so")

ABI_VERSION = 1
NOALLOC_SCRATCH_BYTES = 64 << 20  # ARGUS_NOALLOC_SCRATCH_BYTES
KIND_BEGIN, KIND_END = 1, 2
OUT_INSTANCES, OUT_INSTANCE_EXCL, FORCE_FULL_SORT, FORCE_EVENT_SORT, FORCE_RECORD_RADIX = 1, 2, 4, 8, 16
NUM_COUNTERS = 32
RS_WIDTH = 142
NO_PARENT = 0xFFFFFFFF
UNCLOSED = 0xFFFF
ERRORS = {0: "OK", -1: "ARGUS_E_INVAL", -2: "ARGUS_E_ABI", -3: "ARGUS_E_ALIGN",
          -4: "ARGUS_E_CAPACITY", -5: "ARGUS_E_DEVICE", -6: "ARGUS_E_HIP", -7: "ARGUS_E_IO"}
COUNTER_NAMES = [
    "n_records", "n_valid", "n_bad_kind", "n_bad_region", "n_begin", "n_end",
    "ts_min", "ts_max", "n_ctx", "n_matched", "n_mismatched", "n_unclosed",
    "n_orphan_end", "n_self_nested", "max_level", "n_overlap_skipped",
    "ctx_min", "ctx_max",
]
INSTANCE_DTYPE = np.dtype([
    ("t_begin", "<u8"), ("t_end", "<u8"), ("ctx_key", "<u4"), ("parent", "<u4"),
    ("level", "<u4"), ("region_id", "<u2"), ("end_region_id", "<u2"),
])


# Fields of the device-side plan (struct DevPlan in csrc/internal.h) read back
# for measurement: name -> (byte offset, type).  internal.h asserts the same
# offsets, and a test checks that the two agree.
PLAN_BYTES = 1728
PLAN_FIELDS = {
    "n_records": (0, "<u8"), "n_valid": (8, "<u8"), "n_begin": (16, "<u8"),
    "rec_ts_bits": (48, "<u4"), "rec_ctx_bits": (52, "<u4"), "rec_wide": (56, "<u4"),
    "unsorted": (104, "<u4"), "n_ev": (128, "<u8"), "rec_slots": (144, "slots"),
    "ev_slots": (784, "slots"), "ev_merge": (1432, "<u4"), "merge_rounds": (1440, "<u4"),
    "merge_end": (1448, "<u8"), "runs": (1712, "<u4"), "n_runs": (1720, "<u8"),
}
# C names of the fields above, as internal.h spells them
PLAN_C_NAMES = {
    "rec_ts_bits": "rec.ts_bits", "rec_ctx_bits": "rec.ctx_bits", "rec_wide": "rec.wide",
    "rec_slots": "rs", "ev_slots": "es", "merge_rounds": "m_rounds", "merge_end": "m_end",
}
_SLOT = np.dtype([("active", "<u4"), ("pos", "<u4"), ("src", "<u4"), ("dst", "<u4"),
                  ("lb", "<u4"), ("n_out", "<u4"), ("n_elems", "<u8"), ("tiles", "<u8")])
assert _SLOT.itemsize == 40


class argus_attr_config(ctypes.Structure):
    _fields_ = [("abi_version", ctypes.c_uint32), ("num_regions", ctypes.c_uint32),
                ("num_classes", ctypes.c_uint32), ("group_shift", ctypes.c_uint32),
                ("num_groups", ctypes.c_uint32), ("flags", ctypes.c_uint32),
                ("max_records", ctypes.c_uint64), ("d_region_class", ctypes.c_void_p)]


class argus_attr_outputs(ctypes.Structure):
    _fields_ = [("d_counters", ctypes.c_void_p), ("d_region_stats", ctypes.c_void_p),
                ("d_overlap_group", ctypes.c_void_p), ("d_overlap_global", ctypes.c_void_p),
                ("d_instances", ctypes.c_void_p), ("d_instance_excl", ctypes.c_void_p)]


class argus_samples_config(ctypes.Structure):
    _fields_ = [("abi_version", ctypes.c_uint32), ("num_regions", ctypes.c_uint32),
                ("num_pcs", ctypes.c_uint32), ("num_metrics", ctypes.c_uint32)]


class argus_samples_io(ctypes.Structure):
    _fields_ = [("d_instances", ctypes.c_void_p), ("d_n_instances", ctypes.c_void_p),
                ("max_instances", ctypes.c_uint64), ("d_samples", ctypes.c_void_p),
                ("n_samples", ctypes.c_uint64), ("d_weights", ctypes.c_void_p),
                ("d_metrics", ctypes.c_void_p), ("d_counters", ctypes.c_void_p),
                ("d_n", ctypes.c_void_p), ("d_alpha", ctypes.c_void_p),
                ("d_pc_total", ctypes.c_void_p), ("d_pc_owners", ctypes.c_void_p),
                ("d_entropy", ctypes.c_void_p), ("d_region_total", ctypes.c_void_p),
                ("d_mhat", ctypes.c_void_p)]


class argus_scope(ctypes.Structure):
    _fields_ = [(k, ctypes.c_uint32) for k in ("role_mask", "role_lo", "role_hi", "group_shift",
                                               "group_lo", "group_hi", "iter_lo", "iter_hi")]


class argus_scope_config(ctypes.Structure):
    _fields_ = [("abi_version", ctypes.c_uint32), ("num_regions", ctypes.c_uint32),
                ("scope", argus_scope)]


class argus_scope_io(ctypes.Structure):
    _fields_ = [("d_instances", ctypes.c_void_p), ("d_instance_excl", ctypes.c_void_p),
                ("d_n_instances", ctypes.c_void_p), ("max_instances", ctypes.c_uint64),
                ("d_region_mask", ctypes.c_void_p), ("d_ordinal", ctypes.c_void_p),
                ("d_stats", ctypes.c_void_p), ("d_counters", ctypes.c_void_p)]


class argus_probes_config(ctypes.Structure):
    _fields_ = [("abi_version", ctypes.c_uint32), ("num_regions", ctypes.c_uint32)]


class argus_probes_io(ctypes.Structure):
    _fields_ = [("d_instances", ctypes.c_void_p), ("d_n_instances", ctypes.c_void_p),
                ("max_instances", ctypes.c_uint64), ("d_probes", ctypes.c_void_p),
                ("n_probes", ctypes.c_uint64), ("d_ref", ctypes.c_void_p),
                ("d_completion", ctypes.c_void_p), ("d_groups", ctypes.c_void_p),
                ("d_mean", ctypes.c_void_p), ("d_counters", ctypes.c_void_p)]


PROBE_DTYPE = np.dtype([("t_start", "<u8"), ("t_end", "<u8"), ("ctx_key", "<u4"),
                        ("iteration", "<u4"), ("op_region", "<u2"), ("pad0", "<u2"),
                        ("pad1", "<u4")])
PG_COLUMNS = ["instance", "count", "sum", "issue", "p0", "p20", "p40", "p60", "p80", "p100"]
PR_NUM_COUNTERS = 8
PR_COUNTER_NAMES = ["n_probes", "n_bad", "n_joined", "n_unjoined", "n_groups"]

class argus_handoffs_config(ctypes.Structure):
    _fields_ = [("abi_version", ctypes.c_uint32), ("num_regions", ctypes.c_uint32),
                ("level", ctypes.c_uint32), ("pad", ctypes.c_uint32)]


class argus_handoffs_io(ctypes.Structure):
    _fields_ = [("d_instances", ctypes.c_void_p), ("d_n_instances", ctypes.c_void_p),
                ("max_instances", ctypes.c_uint64), ("d_pairs", ctypes.c_void_p),
                ("d_hist", ctypes.c_void_p), ("d_parent_gap", ctypes.c_void_p),
                ("d_counters", ctypes.c_void_p)]


HO_NUM_COUNTERS = 8
HO_COUNTER_NAMES = ["n_at_level", "n_gaps", "gap_sum"]

class argus_trace_options(ctypes.Structure):
    _fields_ = [("cycles_per_us", ctypes.c_double), ("group_shift", ctypes.c_uint32),
                ("flags", ctypes.c_uint32), ("region_names", ctypes.POINTER(ctypes.c_char_p)),
                ("num_regions", ctypes.c_uint32), ("pad", ctypes.c_uint32)]


TRACE_UNMATCHED = 1

ALL_SCOPE = dict(role_mask=0, role_lo=0, role_hi=0, group_shift=32, group_lo=0, group_hi=0,
                 iter_lo=0, iter_hi=0xFFFFFFFF)
SC_NUM_COUNTERS = 8
SC_COUNTER_NAMES = ["n_instances", "n_in_scope", "n_matched", "n_mismatched", "n_unclosed",
                    "n_self_nested", "n_iterations"]
S_NUM_COUNTERS = 8
S_COUNTER_NAMES = ["n_samples", "n_bad_pc", "w_total", "w_attributed", "w_unattributed",
                   "w_inner_unmatched", "n_pairs", "w_bad_instance"]
SAMPLE_DTYPE = np.dtype([("ts", "<u8"), ("ctx_key", "<u4"), ("pc", "<u4")])

assert ctypes.sizeof(argus_attr_config) == 40
assert ctypes.sizeof(argus_samples_config) == 16
assert ctypes.sizeof(argus_samples_io) == 120
assert ctypes.sizeof(argus_scope_config) == 40
assert ctypes.sizeof(argus_scope_io) == 64
assert ctypes.sizeof(argus_probes_config) == 8
assert ctypes.sizeof(argus_probes_io) == 80
assert PROBE_DTYPE.itemsize == 32
assert ctypes.sizeof(argus_handoffs_config) == 16
assert ctypes.sizeof(argus_handoffs_io) == 56
assert ctypes.sizeof(argus_trace_options) == 32
assert ctypes.sizeof(argus_attr_outputs) == 48

_lib = None


def load_library(path: str = LIB_PATH):
    """Load libargus_attr.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2609_12299_amd.build`"
                           " (the HIP library is required; there is no CPU fallback)")
    lib = ctypes.CDLL(path)
    vp, u64, i32 = ctypes.c_void_p, ctypes.c_uint64, ctypes.c_int
    lib.argus_attr_create.argtypes = [ctypes.POINTER(argus_attr_config), ctypes.POINTER(vp)]
    lib.argus_attr_create.restype = i32
    lib.argus_attr_workspace_bytes.argtypes = [vp, u64]
    lib.argus_attr_workspace_bytes.restype = ctypes.c_size_t
    lib.argus_attr_run.argtypes = [vp, vp, u64, vp, ctypes.c_size_t,
                                   ctypes.POINTER(argus_attr_outputs), vp]
    lib.argus_attr_run.restype = i32
    lib.argus_attr_run_noalloc.argtypes = [vp, vp, u64, ctypes.POINTER(argus_attr_outputs), vp]
    lib.argus_attr_run_noalloc.restype = i32
    lib.argus_attr_samples.argtypes = [ctypes.POINTER(argus_samples_config),
                                       ctypes.POINTER(argus_samples_io), vp]
    lib.argus_attr_samples.restype = i32
    lib.argus_attr_scope_workspace_bytes.argtypes = [u64]
    lib.argus_attr_scope_workspace_bytes.restype = ctypes.c_size_t
    lib.argus_attr_scope.argtypes = [ctypes.POINTER(argus_scope_config),
                                     ctypes.POINTER(argus_scope_io), vp, ctypes.c_size_t, vp]
    lib.argus_attr_scope.restype = i32
    lib.argus_attr_probes_workspace_bytes.argtypes = [u64, u64]
    lib.argus_attr_probes_workspace_bytes.restype = ctypes.c_size_t
    lib.argus_attr_probes.argtypes = [ctypes.POINTER(argus_probes_config),
                                      ctypes.POINTER(argus_probes_io), vp, ctypes.c_size_t, vp]
    lib.argus_attr_probes.restype = i32
    lib.argus_attr_handoffs_workspace_bytes.argtypes = [u64, ctypes.c_uint32]
    lib.argus_attr_handoffs_workspace_bytes.restype = ctypes.c_size_t
    lib.argus_attr_handoffs.argtypes = [ctypes.POINTER(argus_handoffs_config),
                                        ctypes.POINTER(argus_handoffs_io), vp, ctypes.c_size_t, vp]
    lib.argus_attr_handoffs.restype = i32
    lib.argus_attr_chrome_trace.argtypes = [vp, u64, vp, vp, u64,
                                            ctypes.POINTER(argus_trace_options), ctypes.c_char_p]
    lib.argus_attr_chrome_trace.restype = i32
    lib.argus_attr_destroy.argtypes = [vp]
    lib.argus_attr_destroy.restype = None
    lib.argus_attr_last_error.argtypes = [vp]
    lib.argus_attr_last_error.restype = ctypes.c_char_p
    lib.argus_attr_set_timing.argtypes = [vp, i32]
    lib.argus_attr_set_timing.restype = i32
    lib.argus_attr_kernel_times.argtypes = [vp, ctypes.POINTER(ctypes.c_char_p),
                                            ctypes.POINTER(ctypes.c_float), i32]
    lib.argus_attr_kernel_times.restype = i32
    lib.argus_attr_set_timing_filter.argtypes = [vp, ctypes.c_char_p]
    lib.argus_attr_set_timing_filter.restype = i32
    _lib = lib
    return lib


# ------------------------------------------------------------ C ABI, 1:1

def argus_attr_create(cfg: argus_attr_config):
    """Returns (code, handle)."""
    h = ctypes.c_void_p()
    rc = load_library().argus_attr_create(ctypes.byref(cfg), ctypes.byref(h))
    return rc, h


def argus_attr_workspace_bytes(h, n_records: int) -> int:
    return load_library().argus_attr_workspace_bytes(h, n_records)


def argus_attr_run(h, d_records: int, n_records: int, d_workspace: int, workspace_bytes: int,
                   out: argus_attr_outputs, stream: int) -> int:
    return load_library().argus_attr_run(h, d_records, n_records, d_workspace, workspace_bytes,
                                         ctypes.byref(out), stream)


def argus_attr_run_noalloc(h, d_records: int, n_records: int, out: argus_attr_outputs,
                           stream: int) -> int:
    return load_library().argus_attr_run_noalloc(h, d_records, n_records,
                                                 ctypes.byref(out) if out is not None else None,
                                                 stream)


def argus_attr_samples(cfg: argus_samples_config, io: argus_samples_io, stream: int) -> int:
    return load_library().argus_attr_samples(ctypes.byref(cfg) if cfg is not None else None,
                                             ctypes.byref(io) if io is not None else None, stream)


def attribute_samples(instances, n_instances, samples, num_regions: int, num_pcs: int,
                      weights=None, metrics=None, stream=None) -> dict:
    """argus_attr_samples on torch CUDA tensors.

    instances: the instance tensor argus_attr_run wrote (uint8 [cap, 32]);
    n_instances: a 1-element uint64 CUDA tensor holding the instance count
    (e.g. counters[4:5] of that run); samples: uint8 [S, 16] (or any 16-byte
    records); weights: uint32 [S] or None; metrics: float64 [M, P] or None.
    Returns the output tensors (valid once the stream has completed)."""
    import torch
    dev = samples.device
    R, P = int(num_regions), int(num_pcs)
    M = 0 if metrics is None else int(metrics.shape[0])
    ns = samples.numel() * samples.element_size() // 16
    cap = instances.numel() * instances.element_size() // 32
    out = dict(counters=torch.empty(S_NUM_COUNTERS, dtype=torch.uint64, device=dev),
               n=torch.empty((P, R), dtype=torch.uint64, device=dev),
               alpha=torch.empty((P, R), dtype=torch.float64, device=dev),
               pc_total=torch.empty(P, dtype=torch.uint64, device=dev),
               pc_owners=torch.empty(P, dtype=torch.uint32, device=dev),
               entropy=torch.empty(P, dtype=torch.float64, device=dev),
               region_total=torch.empty(R, dtype=torch.uint64, device=dev),
               mhat=torch.empty((M, R), dtype=torch.float64, device=dev))
    cfg = argus_samples_config(ABI_VERSION, R, P, M)
    io = argus_samples_io(instances.data_ptr() if cap else None, n_instances.data_ptr(), cap,
                          samples.data_ptr() if ns else None, ns,
                          weights.data_ptr() if weights is not None else None,
                          metrics.data_ptr() if M else None,
                          out["counters"].data_ptr(), out["n"].data_ptr(),
                          out["alpha"].data_ptr(), out["pc_total"].data_ptr(),
                          out["pc_owners"].data_ptr(), out["entropy"].data_ptr(),
                          out["region_total"].data_ptr(), out["mhat"].data_ptr() if M else None)
    s = stream if stream is not None else torch.cuda.current_stream(dev)
    rc = argus_attr_samples(cfg, io, s.cuda_stream)
    if rc != 0:
        raise ArgusError(rc, "argus_attr_samples rejected its arguments")
    return out


def argus_attr_scope_workspace_bytes(max_instances: int) -> int:
    return load_library().argus_attr_scope_workspace_bytes(max_instances)


def argus_attr_scope(cfg: argus_scope_config, io: argus_scope_io, d_workspace: int,
                     workspace_bytes: int, stream: int) -> int:
    return load_library().argus_attr_scope(ctypes.byref(cfg) if cfg is not None else None,
                                           ctypes.byref(io) if io is not None else None,
                                           d_workspace, workspace_bytes, stream)


def scope_statistics(instances, instance_excl, n_instances, num_regions: int, region_mask=None,
                     stream=None, **scope) -> dict:
    """argus_attr_scope on torch CUDA tensors: the instance and exclusive-time
    tensors argus_attr_run wrote, `n_instances` a 1-element uint64 CUDA
    tensor (e.g. counters[4:5]); scope fields as keyword arguments (default:
    everything).  Returns ordinal [cap] u32 (the first n valid), stats
    [R, 142] u64 and counters [8] u64 (valid once the stream completes)."""
    import torch
    dev = instances.device
    cap = instances.numel() * instances.element_size() // 32
    R = int(num_regions)
    f = dict(ALL_SCOPE)
    f.update(scope)
    cfg = argus_scope_config(ABI_VERSION, R, argus_scope(**{k: int(v) for k, v in f.items()}))
    out = dict(ordinal=torch.empty(max(cap, 1), dtype=torch.uint32, device=dev),
               stats=torch.empty((R, RS_WIDTH), dtype=torch.uint64, device=dev),
               counters=torch.empty(SC_NUM_COUNTERS, dtype=torch.uint64, device=dev))
    need = argus_attr_scope_workspace_bytes(cap)
    ws = torch.empty(need + 256, dtype=torch.uint8, device=dev)
    ws_ptr = (ws.data_ptr() + 255) & ~255
    io = argus_scope_io(instances.data_ptr() if cap else None,
                        instance_excl.data_ptr() if cap else None, n_instances.data_ptr(), cap,
                        region_mask.data_ptr() if region_mask is not None else None,
                        out["ordinal"].data_ptr(), out["stats"].data_ptr(),
                        out["counters"].data_ptr())
    s = stream if stream is not None else torch.cuda.current_stream(dev)
    rc = argus_attr_scope(cfg, io, ws_ptr, need, s.cuda_stream)
    if rc != 0:
        raise ArgusError(rc, "argus_attr_scope rejected its arguments")
    out["_workspace"] = ws  # keeps the workspace alive until the caller drops the result
    return out


def argus_attr_probes_workspace_bytes(max_instances: int, n_probes: int) -> int:
    return load_library().argus_attr_probes_workspace_bytes(max_instances, n_probes)


def argus_attr_probes(cfg: argus_probes_config, io: argus_probes_io, d_workspace: int,
                      workspace_bytes: int, stream: int) -> int:
    return load_library().argus_attr_probes(ctypes.byref(cfg) if cfg is not None else None,
                                            ctypes.byref(io) if io is not None else None,
                                            d_workspace, workspace_bytes, stream)


def join_probes(instances, n_instances, probes, num_regions: int, stream=None) -> dict:
    """argus_attr_probes on torch CUDA tensors: the reference instance tensor
    argus_attr_run wrote, `n_instances` a 1-element uint64 CUDA tensor
    (e.g. counters[4:5]) and the probes (uint8 [P, 32] or any 32-byte
    records).  Returns ref [P] u32, completion [P] u64, groups [P, 10] u64,
    mean [P] f64 (the first counters[4] groups valid) and counters [8] u64."""
    import torch
    dev = probes.device
    cap = instances.numel() * instances.element_size() // 32
    npr = probes.numel() * probes.element_size() // 32
    out = dict(ref=torch.empty(max(npr, 1), dtype=torch.uint32, device=dev),
               completion=torch.empty(max(npr, 1), dtype=torch.uint64, device=dev),
               groups=torch.empty((max(npr, 1), 10), dtype=torch.uint64, device=dev),
               mean=torch.empty(max(npr, 1), dtype=torch.float64, device=dev),
               counters=torch.empty(PR_NUM_COUNTERS, dtype=torch.uint64, device=dev))
    need = argus_attr_probes_workspace_bytes(cap, npr)
    ws = torch.empty(need + 256, dtype=torch.uint8, device=dev)
    ws_ptr = (ws.data_ptr() + 255) & ~255
    cfg = argus_probes_config(ABI_VERSION, int(num_regions))
    io = argus_probes_io(instances.data_ptr() if cap else None, n_instances.data_ptr(), cap,
                         probes.data_ptr() if npr else None, npr, out["ref"].data_ptr(),
                         out["completion"].data_ptr(), out["groups"].data_ptr(),
                         out["mean"].data_ptr(), out["counters"].data_ptr())
    s = stream if stream is not None else torch.cuda.current_stream(dev)
    rc = argus_attr_probes(cfg, io, ws_ptr, need, s.cuda_stream)
    if rc != 0:
        raise ArgusError(rc, "argus_attr_probes rejected its arguments")
    out["_workspace"] = ws
    return out


def argus_attr_handoffs_workspace_bytes(max_instances: int, num_regions: int) -> int:
    return load_library().argus_attr_handoffs_workspace_bytes(max_instances, num_regions)


def argus_attr_handoffs(cfg: argus_handoffs_config, io: argus_handoffs_io, d_workspace: int,
                        workspace_bytes: int, stream: int) -> int:
    return load_library().argus_attr_handoffs(ctypes.byref(cfg) if cfg is not None else None,
                                              ctypes.byref(io) if io is not None else None,
                                              d_workspace, workspace_bytes, stream)


def phase_handoffs(instances, n_instances, num_regions: int, level: int = 0,
                   parent_gap: bool = True, stream=None) -> dict:
    """argus_attr_handoffs on torch CUDA tensors (the instance tensor
    argus_attr_run wrote and a 1-element uint64 CUDA tensor with the instance
    count).  Returns pairs [R, R, 4] u64, hist [65] u64, parent_gap [cap]
    u64 (if asked) and counters [8] u64."""
    import torch
    dev = instances.device
    cap = instances.numel() * instances.element_size() // 32
    R = int(num_regions)
    out = dict(pairs=torch.empty((R, R, 4), dtype=torch.uint64, device=dev),
               hist=torch.empty(65, dtype=torch.uint64, device=dev),
               counters=torch.empty(HO_NUM_COUNTERS, dtype=torch.uint64, device=dev))
    if parent_gap:
        out["parent_gap"] = torch.empty(max(cap, 1), dtype=torch.uint64, device=dev)
    need = argus_attr_handoffs_workspace_bytes(cap, R)
    ws = torch.empty(need + 256, dtype=torch.uint8, device=dev)
    ws_ptr = (ws.data_ptr() + 255) & ~255
    cfg = argus_handoffs_config(ABI_VERSION, R, int(level), 0)
    io = argus_handoffs_io(instances.data_ptr() if cap else None, n_instances.data_ptr(), cap,
                           out["pairs"].data_ptr(), out["hist"].data_ptr(),
                           out["parent_gap"].data_ptr() if parent_gap else None,
                           out["counters"].data_ptr())
    s = stream if stream is not None else torch.cuda.current_stream(dev)
    rc = argus_attr_handoffs(cfg, io, ws_ptr, need, s.cuda_stream)
    if rc != 0:
        raise ArgusError(rc, "argus_attr_handoffs rejected its arguments")
    out["_workspace"] = ws
    return out


def argus_attr_chrome_trace(instances: np.ndarray, path: str, num_regions: int,
                            cycles_per_us: float, group_shift: int = 0, groups=None, mean=None,
                            region_names=None, unmatched: bool = False) -> int:
    """Write the Chrome-trace JSON of host instances (INSTANCE_DTYPE) and,
    optionally, probe groups (u64 [G, 10]) with their means (f64 [G])."""
    inst = np.ascontiguousarray(instances)
    n = inst.nbytes // 32
    g = None if groups is None else np.ascontiguousarray(groups, dtype=np.uint64).reshape(-1, 10)
    m = None if mean is None else np.ascontiguousarray(mean, dtype=np.float64)
    ng = 0 if g is None else g.shape[0]
    names = None
    if region_names is not None:
        names = (ctypes.c_char_p * len(region_names))(*[x.encode() for x in region_names])
    opt = argus_trace_options(float(cycles_per_us), int(group_shift),
                              TRACE_UNMATCHED if unmatched else 0,
                              ctypes.cast(names, ctypes.POINTER(ctypes.c_char_p)) if names else None,
                              int(num_regions), 0)
    return load_library().argus_attr_chrome_trace(
        inst.ctypes.data if n else None, n, g.ctypes.data if ng else None,
        m.ctypes.data if ng else None, ng, ctypes.byref(opt), path.encode())


def argus_attr_destroy(h) -> None:
    load_library().argus_attr_destroy(h)


def argus_attr_last_error(h) -> str:
    s = load_library().argus_attr_last_error(h)
    return s.decode() if s else ""


def argus_attr_set_timing(h, enable: bool) -> int:
    return load_library().argus_attr_set_timing(h, 1 if enable else 0)


def argus_attr_set_timing_filter(h, name) -> int:
    return load_library().argus_attr_set_timing_filter(h, name.encode() if name else None)


def argus_attr_kernel_times(h, cap: int = 1 << 16):
    """[(name, ms)] for every launch of every timed run since the last call."""
    names = (ctypes.c_char_p * cap)()
    ms = (ctypes.c_float * cap)()
    n = load_library().argus_attr_kernel_times(h, names, ms, cap)
    if n < 0:
        raise RuntimeError(f"argus_attr_kernel_times failed: {ERRORS.get(n, n)}")
    return [(names[i].decode(), float(ms[i])) for i in range(min(n, cap))]


class ArgusError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{ERRORS.get(code, code)}: {msg}")
        self.code = code


# ------------------------------------------------------------ torch wrapper

class RegionAttribution:
    """Region attribution on one GPU.

    records: a CUDA tensor of uint8 [N, 16] (or any dtype whose bytes are the
    16-byte records), 16-byte aligned.  region_class: sequence or tensor of R
    class ids (>= num_classes: unclassified).
    """

    def __init__(self, num_regions: int, num_classes: int = 0, region_class=None,
                 group_shift: int = 0, num_groups: int = 0, max_records: int = 1 << 20,
                 instances: bool = True, instance_excl: bool = True,
                 force_full_sort: bool = False, force_event_sort: bool = False,
                 force_record_radix: bool = False, device=None):
        import torch
        self.torch = torch
        self.device = torch.device(device if device is not None else "cuda")
        self.R, self.K, self.G = int(num_regions), int(num_classes), int(num_groups)
        if self.K > 0:
            rc = torch.as_tensor(np.asarray(region_class, dtype=np.uint8), device=self.device)
            self.region_class = rc.contiguous()
            rc_ptr = self.region_class.data_ptr()
        else:
            self.region_class, rc_ptr = None, None
        flags = (OUT_INSTANCES if instances else 0) | (OUT_INSTANCE_EXCL if instance_excl else 0)
        flags |= FORCE_FULL_SORT if force_full_sort else 0
        flags |= FORCE_EVENT_SORT if force_event_sort else 0
        flags |= FORCE_RECORD_RADIX if force_record_radix else 0
        self.flags = flags
        self.cfg = argus_attr_config(ABI_VERSION, self.R, self.K, int(group_shift),
                                     self.G if self.K else 0, flags, int(max_records), rc_ptr)
        rc, self.h = argus_attr_create(self.cfg)
        if rc != 0:
            raise ArgusError(rc, "argus_attr_create rejected the configuration")
        self._ws = None

    def close(self):
        if getattr(self, "h", None):
            argus_attr_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:  # noqa: BLE001 - interpreter shutdown
            pass

    def alloc(self, n: int) -> dict:
        """Output tensors for up to n records."""
        t = self.torch
        d = self.device
        out = dict(
            counters=t.zeros(NUM_COUNTERS, dtype=t.uint64, device=d),
            region_stats=t.zeros((self.R, RS_WIDTH), dtype=t.uint64, device=d),
        )
        if self.K:
            out["overlap_group"] = t.zeros((self.G, 2, self.K, self.K), dtype=t.uint64, device=d)
            out["overlap_global"] = t.zeros((2, self.K, self.K), dtype=t.uint64, device=d)
        if self.flags & OUT_INSTANCES:
            out["instances"] = t.zeros((max(n, 1), 32), dtype=t.uint8, device=d)
        if self.flags & OUT_INSTANCE_EXCL:
            out["instance_excl"] = t.zeros(max(n, 1), dtype=t.uint64, device=d)
        return out

    def workspace(self, n: int):
        need = argus_attr_workspace_bytes(self.h, n)
        if need == 0:
            raise ArgusError(-4, "n exceeds max_records")
        if self._ws is None or self._ws.numel() < need + 256:
            self._ws = None
            self._ws = self.torch.empty(need + 256, dtype=self.torch.uint8, device=self.device)
        base = self._ws.data_ptr()
        aligned = (base + 255) & ~255
        return aligned, need

    def _outputs(self, out: dict) -> argus_attr_outputs:
        return argus_attr_outputs(
            out["counters"].data_ptr(), out["region_stats"].data_ptr(),
            out["overlap_group"].data_ptr() if self.K else None,
            out["overlap_global"].data_ptr() if self.K else None,
            out["instances"].data_ptr() if "instances" in out else None,
            out["instance_excl"].data_ptr() if "instance_excl" in out else None)

    def run(self, records, out: dict | None = None, stream=None) -> dict:
        """Enqueue on `stream` (default: the current torch stream); returns the
        output tensors (valid once the stream has completed)."""
        t = self.torch
        n = records.numel() * records.element_size() // 16
        if out is None:
            out = self.alloc(n)
        ws, ws_bytes = self.workspace(n)
        s = stream if stream is not None else t.cuda.current_stream(self.device)
        rc = argus_attr_run(self.h, records.data_ptr() if n else None, n, ws, ws_bytes,
                            self._outputs(out), s.cuda_stream)
        if rc != 0:
            raise ArgusError(rc, argus_attr_last_error(self.h))
        return out

    def run_noalloc(self, records, out: dict, stream=None) -> dict:
        """argus_attr_run_noalloc: the same run with the library's built-in
        workspace (no workspace tensor); `out` must be preallocated."""
        t = self.torch
        n = records.numel() * records.element_size() // 16
        s = stream if stream is not None else t.cuda.current_stream(self.device)
        rc = argus_attr_run_noalloc(self.h, records.data_ptr() if n else None, n,
                                    self._outputs(out), s.cuda_stream)
        if rc != 0:
            raise ArgusError(rc, argus_attr_last_error(self.h))
        return out

    def plan(self) -> dict:
        """The device-side plan of the last run (read back for measurement:
        which sort passes ran, whether the full sort was needed, the number
        of overlap events).  Synchronises the device."""
        if self._ws is None:
            raise RuntimeError("no run yet")
        t = self.torch
        t.cuda.synchronize(self.device)
        off = ((self._ws.data_ptr() + 255) & ~255) - self._ws.data_ptr()
        raw = self._ws[off:off + PLAN_BYTES].cpu().numpy()
        res = {}
        for name, (at, dt) in PLAN_FIELDS.items():
            if dt == "slots":
                res[name] = raw[at:at + 16 * _SLOT.itemsize].view(_SLOT).copy()
            else:
                res[name] = int(raw[at:at + np.dtype(dt).itemsize].view(dt)[0])
        return res

    def set_timing(self, on: bool):
        rc = argus_attr_set_timing(self.h, on)
        if rc != 0:
            raise ArgusError(rc, argus_attr_last_error(self.h))

    def set_timing_filter(self, name):
        """Time only the launches of one step (None: every launch)."""
        rc = argus_attr_set_timing_filter(self.h, name)
        if rc != 0:
            raise ArgusError(rc, argus_attr_last_error(self.h))

    def kernel_times(self):
        return argus_attr_kernel_times(self.h)


def to_host(out: dict) -> dict:
    """Copy results to numpy; instances become structured arrays trimmed to n_begin."""
    res = {}
    for k, v in out.items():
        a = v.cpu().numpy()
        res[k] = a
    nb = int(res["counters"][4])
    if "instances" in res:
        res["instances"] = res["instances"].reshape(-1).view(INSTANCE_DTYPE)[:nb]
    if "instance_excl" in res:
        res["instance_excl"] = res["instance_excl"][:nb]
    return res
