"""Host-side pieces of bench.py: the algorithmic byte counts behind the
roofline figures and the guard on recorded counter traffic."""
import json
import os

import bench


def test_algorithmic_bytes_per_param():
    # BERT-Large, n = 32, fp32 gradients: worker 1/8 + 32 * (4 + 4 + 4 + 1/8)
    assert bench.algorithmic_bytes_per_param(32) == (388.125, 12.125, 12.125)
    # 16-bit gradients cut 2 bytes per worker row
    w, s, u = bench.algorithmic_bytes_per_param(32, 2)
    assert w == 388.125 - 64 and (s, u) == (12.125, 12.125)
    # the server reads n sign bits per element
    assert bench.algorithmic_bytes_per_param(256)[1] == 256 / 8 + 8.125


def test_measured_traffic_requires_matching_kernel_source(tmp_path, monkeypatch):
    prof = tmp_path / "profiles"
    prof.mkdir()
    src = tmp_path / "paper_2102_02888_amd" / "csrc"
    src.mkdir(parents=True)
    for f in bench.KERNEL_SOURCES:
        (src / f).write_text("// %s\nint v = 1;\n" % f)
    import hashlib
    h = hashlib.sha256()
    for f in bench.KERNEL_SOURCES:
        h.update(b"int v = 1;\0")
    info = {"kernels_source_sha256": h.hexdigest(),
            "kernels": {"k_update": {"traffic_bytes": 123.0}}}
    (prof / "pmc_traffic_w.md").write_text("x\n```json\n%s\n```\n" % json.dumps(info))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.measured_traffic("w", "k_update") == 123.0
    assert bench.measured_traffic("w", "k_other") is None
    assert bench.measured_traffic("missing", "k_update") is None
    # a comment or layout edit keeps the counters, a code change drops them
    (src / "onebit_grid.h").write_text("/* launch shapes */ int v =\n  1; // v2\n")
    assert bench.measured_traffic("w", "k_update") == 123.0
    (src / "onebit_grid.h").write_text("int v = 2;\n")
    assert bench.measured_traffic("w", "k_update") is None


def test_code_text_drops_comments_only():
    src = ('int a; // "x"\n/* b\n c */ const char *s = "// kept /* \\" q";'
           " char q = '/';  x  =\t1 / 2;")
    assert bench.code_text(src) == ('int a; const char *s = "// kept /* \\" q";'
                                    " char q = '/'; x = 1 / 2;")


def test_multi_gpu_request_is_refused():
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_cpu_model_is_named():
    name = bench._cpu_model()
    assert name is None or (isinstance(name, str) and name)


def test_hbm_probe_library_rejects_bad_arguments_on_the_host():
    """The streaming probe's library loads without a GPU and rejects invalid
    arguments before any device call (-1)."""
    import ctypes
    from paper_2102_02888_amd import build, hbm_probe
    if not os.path.exists(hbm_probe.LIB_PATH):
        build.build()
    L = hbm_probe.lib()
    ms = ctypes.c_float()
    fake = ctypes.c_void_p(4096)  # never dereferenced: every call below is rejected first
    assert L.hbm_probe_stream(3, 1, 0, fake, fake, fake, 1024, None, ctypes.byref(ms)) == -1
    assert L.hbm_probe_stream(0, 3, 0, fake, fake, fake, 1024, None, ctypes.byref(ms)) == -1
    assert L.hbm_probe_stream(0, 1, 0, fake, fake, fake, 1000, None, ctypes.byref(ms)) == -1
    assert L.hbm_probe_stream(1, 1, 0, fake, None, fake, 1024, None, ctypes.byref(ms)) == -1
    assert L.hbm_probe_stream(2, 1, 70000, fake, fake, fake, 1024, None, ctypes.byref(ms)) == -1
    assert L.hbm_probe_rowsum(16, 3, fake, 1024, 2, fake, None, ctypes.byref(ms)) == -1
    assert L.hbm_probe_rowsum(16, 2, fake, 1024, 3, fake, None, ctypes.byref(ms)) == -1
    assert L.hbm_probe_rowsum(12, 1, fake, 1024, 2, fake, None, ctypes.byref(ms)) == -1
    assert L.hbm_probe_rowsum(0, 1, fake, 1024, 2, fake, None, ctypes.byref(ms)) == -1
    assert L.hbm_probe_rowsum(8, 2, fake, 1024, 2, fake, None, ctypes.byref(ms)) == -1
