"""C-ABI checks that need no GPU: the library loads, exports every function
include/argus_attr.h declares, and rejects bad arguments with the documented
codes before making any HIP call."""
from __future__ import annotations

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "argus_attr.h")


@pytest.fixture(scope="module")
def lib():
    from paper_2609_12299_amd import attr
    if not os.path.exists(attr.LIB_PATH):
        from paper_2609_12299_amd import build
        build.build()
    return attr


def declared_functions():
    src = open(HEADER).read()
    return sorted(set(re.findall(r"\b(argus_attr_[a-z_]+)\s*\(", src)))


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert "argus_attr_run" in names and len(names) >= 7
    so = lib.load_library()
    for n in names:
        assert hasattr(so, n), f"missing export {n}"


def test_struct_layouts_match_header(lib):
    src = open(HEADER).read()
    assert "ARGUS_ATTR_ABI_VERSION 1u" in src
    assert ctypes.sizeof(lib.argus_attr_config) == 40
    assert ctypes.sizeof(lib.argus_attr_outputs) == 48
    assert lib.INSTANCE_DTYPE.itemsize == 32


def cfg(lib, **kw):
    c = lib.argus_attr_config(1, 4, 0, 0, 0, 0, 1 << 20, None)
    for k, v in kw.items():
        setattr(c, k, v)
    return c


@pytest.mark.parametrize("field,value,code", [
    ("abi_version", 2, -2),
    ("num_regions", 0, -1),
    ("num_regions", 65536, -1),
    ("num_classes", 9, -1),
    ("group_shift", 33, -1),
    ("flags", 32, -1),
    ("max_records", 1 << 31, -4),
])
def test_create_rejects_bad_config(lib, field, value, code):
    rc, h = lib.argus_attr_create(cfg(lib, **{field: value}))
    assert rc == code
    assert not h.value


def test_create_requires_class_table_and_groups(lib):
    rc, _ = lib.argus_attr_create(cfg(lib, num_classes=2, num_groups=4))
    assert rc == -1  # d_region_class is NULL
    rc, _ = lib.argus_attr_create(cfg(lib, num_classes=2, num_groups=0, d_region_class=0x1000))
    assert rc == -1


def test_workspace_bytes(lib):
    rc, h = lib.argus_attr_create(cfg(lib))
    assert rc == 0
    try:
        a = lib.argus_attr_workspace_bytes(h, 1000)
        b = lib.argus_attr_workspace_bytes(h, 100000)
        assert 0 < a < b and a % 256 == 0 and b % 256 == 0
        assert lib.argus_attr_workspace_bytes(h, (1 << 20) + 1) == 0
        assert lib.argus_attr_workspace_bytes(None, 10) == 0
    finally:
        lib.argus_attr_destroy(h)


def test_run_argument_errors_before_any_gpu_call(lib):
    rc, h = lib.argus_attr_create(cfg(lib, flags=1))
    assert rc == 0
    try:
        fake = 0x100000  # never dereferenced: every case fails its checks first
        ws = lib.argus_attr_workspace_bytes(h, 64)
        full = lib.argus_attr_outputs(fake, fake, None, None, fake, None)
        no_inst = lib.argus_attr_outputs(fake, fake, None, None, None, None)
        no_counters = lib.argus_attr_outputs(None, fake, None, None, fake, None)
        assert lib.argus_attr_run(None, fake, 64, fake, ws, full, None) == -1
        assert lib.argus_attr_run(h, fake, (1 << 20) + 1, fake, ws, full, None) == -4
        assert lib.argus_attr_run(h, None, 64, fake, ws, full, None) == -1
        assert lib.argus_attr_run(h, fake, 64, fake, ws, no_counters, None) == -1
        assert lib.argus_attr_run(h, fake, 64, fake, ws, no_inst, None) == -1
        assert "d_instances" in lib.argus_attr_last_error(h)
        assert lib.argus_attr_run(h, fake + 8, 64, fake, ws, full, None) == -3
        assert lib.argus_attr_run(h, fake, 64, fake + 16, ws, full, None) == -3
        assert lib.argus_attr_run(h, fake, 64, None, ws, full, None) == -1
        assert lib.argus_attr_run(h, fake, 64, fake, 1024, full, None) == -4
        assert "workspace" in lib.argus_attr_last_error(h)
    finally:
        lib.argus_attr_destroy(h)
    lib.argus_attr_destroy(None)  # no-op


def test_overlap_outputs_required(lib):
    rc, h = lib.argus_attr_create(cfg(lib, num_classes=2, num_groups=4, d_region_class=0x2000))
    assert rc == 0
    try:
        fake = 0x100000
        ws = lib.argus_attr_workspace_bytes(h, 64)
        out = lib.argus_attr_outputs(fake, fake, None, None, None, None)
        assert lib.argus_attr_run(h, fake, 64, fake, ws, out, None) == -1
        assert "overlap" in lib.argus_attr_last_error(h)
    finally:
        lib.argus_attr_destroy(h)


def test_product_path_does_not_touch_the_oracle():
    """The GPU package never imports, links or names the oracle library."""
    pkg = os.path.join(ROOT, "paper_2609_12299_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                text = open(os.path.join(dirpath, f)).read()
                assert "oracle" not in text.lower(), f"{f} mentions the oracle"


def test_noalloc_argument_errors_before_any_gpu_call(lib):
    """The allocation-free entry point checks its arguments, and that the
    run fits its built-in workspace, before making any HIP call."""
    rc, h = lib.argus_attr_create(cfg(lib, flags=1))
    assert rc == 0
    try:
        fake = 0x100000  # never dereferenced: every case fails its checks first
        full = lib.argus_attr_outputs(fake, fake, None, None, fake, None)
        no_inst = lib.argus_attr_outputs(fake, fake, None, None, None, None)
        f = lib.argus_attr_run_noalloc
        assert f(None, fake, 64, full, None) == -1
        assert f(h, fake, (1 << 20) + 1, full, None) == -4
        assert f(h, None, 64, full, None) == -1
        assert f(h, fake, 64, None, None) == -1
        assert f(h, fake, 64, no_inst, None) == -1
        assert f(h, fake + 8, 64, full, None) == -3
        # 2^20 records need more workspace than the built-in array holds
        assert lib.argus_attr_workspace_bytes(h, 1 << 20) > lib.NOALLOC_SCRATCH_BYTES
        assert f(h, fake, 1 << 20, full, None) == -4
        assert "built-in workspace" in lib.argus_attr_last_error(h)
    finally:
        lib.argus_attr_destroy(h)


def test_noalloc_scratch_size_matches_header(lib):
    src = open(HEADER).read()
    m = re.search(r"#define ARGUS_NOALLOC_SCRATCH_BYTES \((\d+)u << (\d+)\)", src)
    assert m and int(m.group(1)) << int(m.group(2)) == lib.NOALLOC_SCRATCH_BYTES


def test_plan_fields_match_internal_layout(lib):
    """The plan fields the binding reads back sit where internal.h asserts them."""
    src = open(os.path.join(ROOT, "paper_2609_12299_amd", "csrc", "internal.h")).read()
    asserted = {m.group(1): int(m.group(2)) for m in
                re.finditer(r"static_assert\(offsetof\(DevPlan, ([a-z_.]+)\) == (\d+)", src)}
    size = re.search(r"static_assert\(sizeof\(DevPlan\) == (\d+)", src)
    assert size and int(size.group(1)) == lib.PLAN_BYTES
    for name, (off, _) in lib.PLAN_FIELDS.items():
        cname = lib.PLAN_C_NAMES.get(name, name)
        assert asserted.get(cname) == off, f"{name} ({cname}): binding {off}, header {asserted.get(cname)}"
