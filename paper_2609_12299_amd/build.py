"""Build the HIP library libargus_attr.so for gfx950 (in-tree).

Run ``python -m paper_2609_12299_amd.build`` or call :func:`build`.  Every
source is compiled every time (the build is the "does it compile" check).
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libargus_attr.so")
SOURCES = ["attr_host.hip", "k_ingest.hip", "k_radix.hip", "k_match.hip", "k_resolve.hip", "k_merge.hip",
           "k_agg.hip", "k_overlap.hip", "k_samples.hip", "k_scope.hip", "trace_export.hip"]
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def flags() -> list[str]:
    return [
        "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
        # no packed-FP32 instructions anywhere in the device code
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        # uniform-address atomics: reduce across the wave with DPP, not with a
        # scalar loop over the active lanes
        "-mllvm", "-amdgpu-atomic-optimizer-strategy=DPP",
        "-Wall", "-Wno-unused-function", "-Wno-unused-variable",
        "-I", os.path.join(HERE, "..", "include"),
    ]


# per-source flags: the sample attribution rounds every product on its own
FILE_FLAGS = {"k_samples.hip": ["-ffp-contract=off"]}


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [hipcc(), *flags(), *FILE_FLAGS.get(src, []), "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr}")
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(len(SOURCES), 8)) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


def resources() -> str:
    """Per-kernel register, scratch, occupancy and LDS use as the compiler
    reports them for gfx950 (device-only compile of every source)."""
    import re
    import tempfile
    rows = []
    keys = ("VGPRs", "AGPRs", "TotalSGPRs", "ScratchSize [bytes/lane]", "Occupancy [waves/SIMD]",
            "LDS Size [bytes/block]", "VGPRs Spill", "SGPRs Spill")
    with tempfile.TemporaryDirectory() as tmp:
        for src in SOURCES:
            cmd = [hipcc(), *flags(), *FILE_FLAGS.get(src, []), "--offload-device-only", "-c",
                   os.path.join(CSRC, src),
                   "-o", os.path.join(tmp, src + ".o"), "-Rpass-analysis=kernel-resource-usage"]
            r = subprocess.run(cmd, capture_output=True, text=True)
            if r.returncode != 0:
                raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr}")
            cur = None
            for line in r.stderr.splitlines():
                m = re.search(r"remark:\s+Function Name: (\S+)", line)
                if m:
                    cur = {"kernel": m.group(1), "file": src}
                    rows.append(cur)
                    continue
                for k in keys:
                    m = re.search(r"remark:\s+" + re.escape(k) + r": (\d+) ", line)
                    if m and cur is not None:
                        cur[k] = int(m.group(1))
    names = [r["kernel"] for r in rows]
    filt = shutil.which("c++filt") or shutil.which("llvm-cxxfilt")
    if filt and names:
        out = subprocess.run([filt], input="\n".join(names), capture_output=True, text=True).stdout
        for r, d in zip(rows, out.splitlines()):
            r["kernel"] = d.split("(")[0]
    head = (f"{'kernel':48s} {'file':14s} VGPR AGPR SGPR spill sspill scratch waves/SIMD   LDS B"
            "\n(spill: VGPRs spilled to scratch; sspill: SGPRs spilled to VGPR lanes)")
    lines = [head]
    for r in rows:
        lines.append(f"{r['kernel'][:48]:48s} {r['file']:14s} {r.get('VGPRs', 0):4d} "
                     f"{r.get('AGPRs', 0):4d} {r.get('TotalSGPRs', 0):4d} {r.get('VGPRs Spill', 0):5d} "
                     f"{r.get('SGPRs Spill', 0):6d} "
                     f"{r.get('ScratchSize [bytes/lane]', 0):7d} "
                     f"{r.get('Occupancy [waves/SIMD]', 0):10d} "
                     f"{r.get('LDS Size [bytes/block]', 0):7d}")
    return "\n".join(lines)


if __name__ == "__main__":
    if len(sys.argv) > 1 and sys.argv[1] == "--resources":
        print(resources())
    else:
        build(verbose=True)
    sys.exit(0)
