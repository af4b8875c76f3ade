"""Comparison helpers for the GPU-vs-oracle parity tests."""
import numpy as np

# Floating-point state must agree within this after the free-running steps.
REL_TOL = 1e-5
ABS_TOL = 1e-6


def host(t):
    """GPU tensor -> numpy (int64 sign words come back as uint64)."""
    a = t.detach().cpu().numpy()
    if a.dtype == np.int64:
        a = a.view(np.uint64)
    return a


def check_fp(name, gpu, ref, rel=REL_TOL, abs_=ABS_TOL, mask=None):
    """Asserts |gpu - ref| <= abs_ + rel |ref| elementwise (NaN matches NaN).
    Returns the fraction of bit-identical elements."""
    g = np.asarray(gpu, np.float32)
    r = np.asarray(ref, np.float32)
    assert g.shape == r.shape, (name, g.shape, r.shape)
    if mask is not None:
        g, r = g[..., mask], r[..., mask]
    nan = np.isnan(g) & np.isnan(r)
    diff = np.abs(g.astype(np.float64) - r.astype(np.float64))
    ok = (diff <= abs_ + rel * np.abs(r.astype(np.float64))) | nan
    if not ok.all():
        idx = np.argwhere(~ok)[:5]
        raise AssertionError("%s: %d of %d outside tolerance; first %s gpu=%s ref=%s"
                             % (name, (~ok).sum(), ok.size, idx.tolist(),
                                [float(g[tuple(i)]) for i in idx],
                                [float(r[tuple(i)]) for i in idx]))
    return float((g.view(np.uint32) == r.view(np.uint32)).mean()) if g.size else 1.0


def check_bits(name, gpu, ref):
    g = np.asarray(gpu).view(np.uint64)
    r = np.asarray(ref).view(np.uint64)
    assert g.shape == r.shape, (name, g.shape, r.shape)
    bad = g != r
    if bad.any():
        idx = np.argwhere(bad)[:5]
        raise AssertionError("%s: %d of %d words differ; first %s" % (name, bad.sum(), bad.size,
                                                                     idx.tolist()))


def check_scales(name, gpu, ref, max_ulp=1):
    """Scales agree within max_ulp units in the last place; returns the number
    of scales that are not bit-identical."""
    g = np.asarray(gpu, np.float32)
    r = np.asarray(ref, np.float32)
    assert g.shape == r.shape
    gi = g.view(np.int32).astype(np.int64)
    ri = r.view(np.int32).astype(np.int64)
    nan = np.isnan(g) & np.isnan(r)
    ulps = np.abs(gi - ri)
    bad = (ulps > max_ulp) & ~nan
    if bad.any():
        idx = np.argwhere(bad)[:5]
        raise AssertionError("%s: %d scales differ by more than %d ulp; first %s gpu=%s ref=%s"
                             % (name, bad.sum(), max_ulp, idx.tolist(),
                                [float(g[tuple(i)]) for i in idx],
                                [float(r[tuple(i)]) for i in idx]))
    return int(((ulps != 0) & ~nan).sum())
