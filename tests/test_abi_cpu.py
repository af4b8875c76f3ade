"""Host-side checks of the C-ABI library (no GPU needed): it loads, exports
every entry point its header declares, and rejects bad arguments before
touching the device."""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "onebit.h")


@pytest.fixture(scope="module")
def native():
    from paper_2102_02888_amd import build
    if not os.path.exists(build.LIB):
        build.build()
    from paper_2102_02888_amd import _native
    return _native


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(onebit_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_entry_points():
    names = declared_functions()
    for required in ["onebit_warmup_adam_step", "onebit_worker_compress",
                     "onebit_server_reduce_compress", "onebit_decompress_update",
                     "onebit_step"]:
        assert required in names


def test_library_exports_every_declared_symbol(native):
    lib = native.lib()
    for name in declared_functions():
        assert hasattr(lib, name), name
    assert set(declared_functions()) == set(native.SIGNATURES)
    out = subprocess.run(["nm", "-D", "--defined-only", native.LIB_PATH],
                         capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r"\bT (onebit_\w+)", out))
    assert exported == set(declared_functions())
    # the product library carries nothing of the oracle
    assert "orc_" not in out


def test_status_strings(native):
    lib = native.lib()
    assert lib.onebit_status_str(0) == b"ONEBIT_OK"
    assert lib.onebit_status_str(-1) == b"ONEBIT_EINVAL"
    assert lib.onebit_status_str(-2) == b"ONEBIT_EALIGN"
    assert lib.onebit_status_str(-3) == b"ONEBIT_EHIP"
    assert lib.onebit_status_str(-4) == b"ONEBIT_ENOMEM"
    assert lib.onebit_status_str(7) == b"ONEBIT_UNKNOWN"


def test_argument_errors_before_device(native):
    lib = native.lib()
    out = ctypes.c_void_p(1)
    numel = (ctypes.c_int64 * 2)(10, 20)
    assert lib.onebit_plan_create(numel, 2, 4, None) == -1
    assert lib.onebit_plan_create(None, 2, 4, ctypes.byref(out)) == -1
    assert out.value is None  # cleared on error
    assert lib.onebit_plan_create(numel, 0, 4, ctypes.byref(out)) == -1
    assert lib.onebit_plan_create(numel, 2, 0, ctypes.byref(out)) == -1
    bad = (ctypes.c_int64 * 2)(10, -1)
    assert lib.onebit_plan_create(bad, 2, 4, ctypes.byref(out)) == -1
    assert b"tensor_numel[1]" in lib.onebit_last_error()
    # sizes that would overflow the layout arithmetic are refused up front
    huge = (ctypes.c_int64 * 2)(10, (1 << 63) - 1)
    assert lib.onebit_plan_create(huge, 2, 4, ctypes.byref(out)) == -1
    assert b"tensor_numel[1] exceeds" in lib.onebit_last_error()
    # K * n segments must fit in int32; refused before any device call
    many = (ctypes.c_int64 * (1 << 20))()
    assert lib.onebit_plan_create(many, 1 << 20, 1 << 12, ctypes.byref(out)) == -1
    assert b"segments" in lib.onebit_last_error()
    for fn in ["onebit_plan_destroy"]:
        assert getattr(lib, fn)(None) == -1
    assert lib.onebit_plan_get_info(None, None) == -1
    assert lib.onebit_decompress_update(None, None, None, None, None, None, 0.0, 0.0, None) == -1
    assert lib.onebit_step(None, *([None] * 4), 0, 0, None, 0, *([None] * 5), 0.0, 0.0, 0.0,
                           None, None) == -1
    assert lib.onebit_worker_compress(None, None, None, None, None, 0, 0, 1, None, 0, None, 0,
                                      None, 0, 0.9, None, None) == -1


def test_binding_fails_loudly_without_library(tmp_path, monkeypatch):
    from paper_2102_02888_amd import _native
    monkeypatch.setattr(_native, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(_native, "_lib", None)
    with pytest.raises(ImportError):
        _native.lib()
