"""MI355X-native region attribution over begin/end marker traces.

The data-parallel core of the evidence join of "Argus: Orchestrating
Cross-Layer GPU Performance Measurements around Semantic Regions"
(arxiv 2609.12299): marker records become region instances with nesting,
per-region duration statistics, class overlap and ambiguity counts, and PC
samples are attributed to those instances, computed by hand-written HIP
kernels for gfx950 behind a C ABI (include/argus_attr.h).
"""
from .attr import (ABI_VERSION, COUNTER_NAMES, FORCE_EVENT_SORT, FORCE_FULL_SORT,
                   FORCE_RECORD_RADIX, INSTANCE_DTYPE, NOALLOC_SCRATCH_BYTES, NUM_COUNTERS,
                   OUT_INSTANCE_EXCL, OUT_INSTANCES, RS_WIDTH, S_COUNTER_NAMES, SAMPLE_DTYPE,
                   ArgusError, RegionAttribution, argus_attr_config, argus_attr_create,
                   argus_attr_destroy, argus_attr_kernel_times, argus_attr_last_error,
                   argus_attr_outputs, argus_attr_run, argus_attr_run_noalloc,
                   argus_attr_samples, argus_attr_set_timing, argus_attr_set_timing_filter,
                   argus_attr_workspace_bytes, argus_samples_config, argus_samples_io,
                   argus_attr_scope, argus_attr_scope_workspace_bytes, argus_scope,
                   argus_scope_config, argus_scope_io, attribute_samples, load_library,
                   scope_statistics, to_host, PROBE_DTYPE, argus_attr_probes,
                   argus_attr_probes_workspace_bytes, argus_probes_config, argus_probes_io,
                   join_probes, argus_attr_handoffs, argus_attr_handoffs_workspace_bytes,
                   argus_handoffs_config, argus_handoffs_io, phase_handoffs,
                   argus_attr_chrome_trace, argus_trace_options)

__all__ = [
    "ABI_VERSION", "COUNTER_NAMES", "FORCE_EVENT_SORT", "FORCE_FULL_SORT", "FORCE_RECORD_RADIX",
    "INSTANCE_DTYPE", "NOALLOC_SCRATCH_BYTES", "NUM_COUNTERS", "OUT_INSTANCE_EXCL",
    "OUT_INSTANCES", "RS_WIDTH", "S_COUNTER_NAMES", "SAMPLE_DTYPE", "ArgusError",
    "RegionAttribution", "argus_attr_config", "argus_attr_create", "argus_attr_destroy",
    "argus_attr_kernel_times", "argus_attr_last_error", "argus_attr_outputs", "argus_attr_run",
    "argus_attr_run_noalloc", "argus_attr_samples", "argus_attr_set_timing",
    "argus_attr_set_timing_filter", "argus_attr_workspace_bytes", "argus_samples_config",
    "argus_samples_io", "attribute_samples", "load_library", "to_host", "argus_attr_scope",
    "argus_attr_scope_workspace_bytes", "argus_scope", "argus_scope_config", "argus_scope_io",
    "scope_statistics", "PROBE_DTYPE", "argus_attr_probes", "argus_attr_probes_workspace_bytes",
    "argus_probes_config", "argus_probes_io", "join_probes", "argus_attr_handoffs",
    "argus_attr_handoffs_workspace_bytes", "argus_handoffs_config", "argus_handoffs_io",
    "phase_handoffs", "argus_attr_chrome_trace", "argus_trace_options",
]
