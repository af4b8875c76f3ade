"""HBM streaming ceilings for the library's access mixes.

A measurement aid next to the library, not part of its path: ctypes over
lib/libhbmprobe.so (built from csrc/hbm_probe.hip by build.py), with device
buffers from torch.  The kernels use the passes' load and store forms; the
mixes are `read` (one stream read), `copy` (one read, one written) and `mix`
(two read, the second rewritten in place: the worker pass's mix), each over
pieces of 1 KB per stream per wave in flight (k) and unused LDS per 4-wave
workgroup (lds), which caps the workgroups per CU.  `rowsum` is the warm-up's
read pattern (R rows summed per 1024-element tile in row order, fp64).

    python -m paper_2102_02888_amd.hbm_probe

prints one line per case; bench.py reports the best rate of each mix.
"""
import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "lib", "libhbmprobe.so")
PEAK_GBPS = 8000.0
KINDS = ("read", "copy", "mix")
STREAMS = {"read": 1, "copy": 2, "mix": 3}
CASES = tuple((k, lds) for lds in (0, 40960, 65536) for k in (1, 2, 4))

_lib = None


def lib():
    """The probe library (raises ImportError when it is not built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError("%s is not built (paper_2102_02888_amd/build.py builds it)"
                              % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
        L.hbm_probe_stream.argtypes = [i32, i32, i32, vp, vp, vp, i64, vp,
                                       ctypes.POINTER(ctypes.c_float)]
        L.hbm_probe_stream.restype = i32
        L.hbm_probe_rowsum.argtypes = [i32, i32, vp, i64, i32, vp, vp,
                                       ctypes.POINTER(ctypes.c_float)]
        L.hbm_probe_rowsum.restype = i32
        _lib = L
    return _lib


def waves_per_cu(lds):
    """Upper bound on the waves per CU of a 4-wave workgroup with lds bytes
    of LDS (160 KB of LDS and 8 waves per SIMD per CU)."""
    return min(8, (160 * 1024) // lds if lds else 8) * 4


def stream_case(kind, k, lds, a, b, sink, stream):
    """(median ms, GB/s) of one case over the float32 device tensors a and b
    (b unused by `read`) and a one-element sink."""
    import torch
    if a.dtype != torch.float32 or not a.is_contiguous() or a.numel() % 1024:
        raise ValueError("a must be a contiguous float32 tensor of a multiple of 1024 floats")
    if kind != "read" and (b is None or b.dtype != torch.float32 or not b.is_contiguous()
                           or b.numel() < a.numel()):
        raise ValueError("b must be a contiguous float32 tensor at least as long as a")
    ms = ctypes.c_float()
    rc = lib().hbm_probe_stream(KINDS.index(kind), k, lds, a.data_ptr(),
                                None if b is None else b.data_ptr(), sink.data_ptr(), a.numel(),
                                stream.cuda_stream, ctypes.byref(ms))
    if rc:
        raise RuntimeError("hbm_probe_stream(%s, k=%d, lds=%d) returned %d" % (kind, k, lds, rc))
    return ms.value, STREAMS[kind] * a.numel() * 4 / (ms.value * 1e-3) / 1e9


def stream_table(a, b, sink, stream):
    """Every (k, lds) case of every mix: a list of dicts."""
    rows = []
    for k, lds in CASES:
        for kind in KINDS:
            ms, gbps = stream_case(kind, k, lds, a, b, sink, stream)
            rows.append({"kind": kind, "k": k, "lds": lds, "ms": ms, "gbps": gbps})
    return rows


def best(rows):
    """The fastest case of each mix."""
    out = {}
    for kind in KINDS:
        r = max((r for r in rows if r["kind"] == kind), key=lambda r: r["gbps"])
        out[kind] = {"gbps": r["gbps"], "frac": r["gbps"] / PEAK_GBPS, "k": r["k"],
                     "lds": r["lds"]}
    return out


def rowsum_case(w, b, g, D, R, out, stream):
    """(median ms, GB/s) of the row-sum pattern over g ([R, D] float32
    rows) into out (D floats)."""
    ms = ctypes.c_float()
    rc = lib().hbm_probe_rowsum(w, b, g.data_ptr(), D, R, out.data_ptr(), stream.cuda_stream,
                                ctypes.byref(ms))
    if rc:
        raise RuntimeError("hbm_probe_rowsum(w=%d, b=%d) returned %d" % (w, b, rc))
    return ms.value, (R + 1) * D * 4 / (ms.value * 1e-3) / 1e9


def main():
    import torch
    dev = torch.device("cuda:0")
    p = torch.cuda.get_device_properties(dev)
    print("device %s (%s), %d CUs" % (p.name, getattr(p, "gcnArchName", "?"),
                                       p.multi_processor_count), flush=True)
    s = torch.cuda.current_stream(dev)
    floats = 1 << 30  # 4 GiB streams, far beyond the 256 MB last-level cache
    a = torch.zeros(floats, dtype=torch.float32, device=dev)
    b = torch.zeros_like(a)
    sink = torch.zeros(1, dtype=torch.float32, device=dev)
    print("read / copy / mix over %d MiB streams" % (floats * 4 >> 20), flush=True)
    for r in stream_table(a, b, sink, s):
        wpc = waves_per_cu(r["lds"])
        inflight = wpc // 4 * r["k"] * (2 if r["kind"] == "mix" else 1)
        print("%-4s K=%d lds=%5d (<= %2d waves/CU, <= %2d KB/SIMD of loads in flight)  %8.3f ms"
              "  %6.0f GB/s  %.3f" % (r["kind"], r["k"], r["lds"], wpc, inflight, r["ms"],
                                       r["gbps"], r["gbps"] / PEAK_GBPS), flush=True)
    del a, b
    torch.cuda.empty_cache()
    R, D = 32, 334088192  # the BERT-Large shape: 326,258 tiles of 1024
    g = torch.zeros((R, D), dtype=torch.float32, device=dev)
    out = torch.zeros(D, dtype=torch.float32, device=dev)
    print("rowsum over %d rows of %d floats (%.1f GB read)" % (R, D, R * D * 4 / 1e9), flush=True)
    for w, bb in ((16, 1), (16, 2), (8, 1), (4, 1)):
        ms, gbps = rowsum_case(w, bb, g, D, R, out, s)
        print("rowsum R=%d W=%2d B=%d  %8.3f ms  %6.0f GB/s  %.3f"
              % (R, w, bb, ms, gbps, gbps / PEAK_GBPS), flush=True)
    ms, gbps = stream_case("read", 4, 0, g.view(-1), None, sink, s)
    print("flat read of the %d rows  %8.3f ms  %6.0f GB/s  %.3f"
          % (R, ms, gbps, gbps / PEAK_GBPS), flush=True)
    print("done", flush=True)


if __name__ == "__main__":
    main()
