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


# ---------------------------------------------------------------------------
# The oracle on sampled whole segments, run on the host's cores
# ---------------------------------------------------------------------------

def host_threads():
    """Worker threads for the oracle: the process's CPU share, at most 16."""
    import os
    return max(1, min(16, len(os.sched_getaffinity(0))))


class SegmentOracle:
    """Free-running oracle state of a few whole segments of a plan.

    Each segment (tensor k, chunk j) is an independent parameter-server
    problem, so its history needs only its own slice of every input.  The
    oracle library releases the GIL, so the n workers' passes of all sampled
    segments run in parallel threads; each segment's chunk-owner step and
    update follow once its workers are done.  Nothing here computes: every
    step is the oracle's own function."""

    def __init__(self, layout, segs, x_host, n_workers):
        import threading
        from concurrent.futures import ThreadPoolExecutor
        self.n = n_workers
        self.segs = []
        for q in segs:
            b, e = int(layout.seg_begin[q]), int(layout.seg_end[q])
            assert e > b, q
            ln, nw = e - b, (e - b + 63) // 64
            self.segs.append(dict(
                q=q, b=b, e=e, ln=ln, x=np.array(x_host(b, e), np.float32),
                m=np.zeros(ln, np.float32), v=np.zeros(ln, np.float32),
                delta=np.zeros((n_workers, ln), np.float32), dbar=np.zeros(ln, np.float32),
                wbits=np.zeros((n_workers, nw), np.uint64), wscales=np.zeros(n_workers, np.float32),
                sbits=np.zeros(nw, np.uint64), sscale=np.float32(0)))
        self.pool = ThreadPoolExecutor(max_workers=host_threads())
        self._local = threading.local()
        self._maxlen = max(sg["ln"] for sg in self.segs)

    def _scratch(self):
        z = getattr(self._local, "z", None)
        if z is None:
            z = self._local.z = np.zeros(self._maxlen, np.float32)
        return z

    def close(self):
        self.pool.shutdown()

    def warmup(self, grads, t, lr, beta1, beta2, eps, bias_correction=0):
        """grads(b, e) -> [n_grads, e - b] float32 of this step."""
        import oracle
        futs = []
        for sg in self.segs:
            g = np.ascontiguousarray(grads(sg["b"], sg["e"]), np.float32)
            futs.append(self.pool.submit(oracle.warmup_range, 0, sg["ln"], sg["x"], sg["m"],
                                         sg["v"], g, sg["ln"], g.shape[0], lr, beta1, beta2,
                                         eps, bias_correction, t))
        for f in futs:
            f.result()

    def _worker(self, sg, i, g_i, beta1):
        import oracle
        sg["wscales"][i] = oracle.worker_segment(0, sg["ln"], beta1, sg["m"], g_i,
                                                 sg["delta"][i], sg["wbits"][i], self._scratch())

    def _owner(self, sg, received):
        import oracle
        if received is None:
            bits, scales, n = sg["wbits"], sg["wscales"], self.n
        else:
            bits, scales = received
            n = bits.shape[0]
        sg["sscale"] = oracle.server_segment(0, sg["ln"], n, np.ascontiguousarray(bits).reshape(-1),
                                             bits.shape[1], np.ascontiguousarray(scales), 1,
                                             sg["dbar"], sg["sbits"], self._scratch())

    def _update(self, sg, bits, scale, lr, eps):
        import oracle
        oracle.update_segment(0, sg["ln"], bits, scale, lr, eps, sg["x"], sg["m"], sg["v"])

    def workers(self, grads, beta1):
        """Every local worker's pass (Algorithm 1: momentum, error
        compensation, compression) on every sampled segment."""
        futs = []
        for sg in self.segs:
            g = np.ascontiguousarray(grads(sg["b"], sg["e"]), np.float32)
            futs += [self.pool.submit(self._worker, sg, i, g[i], beta1) for i in range(self.n)]
        for f in futs:
            f.result()

    def owners_and_updates(self, lr, eps, received=None, gathered=None):
        """The chunk owners' average and recompression, then the update, on
        every sampled segment.  received: {q: (bits [rows, words], scales
        [rows])} replaces the local workers' messages of segment q by
        incoming ones; gathered: {q: (bits [words], scale)} gives segment q's
        server message instead of running its owner (a chunk owned by
        another GPU)."""
        received, gathered = received or {}, gathered or {}

        def one(sg):
            if sg["q"] in gathered:
                bits, scale = gathered[sg["q"]]
                sg["sbits"][:] = bits
                sg["sscale"] = np.float32(scale)
            else:
                self._owner(sg, received.get(sg["q"]))
            self._update(sg, sg["sbits"], sg["sscale"], lr, eps)

        for f in [self.pool.submit(one, sg) for sg in self.segs]:
            f.result()

    def step(self, grads, lr, beta1, eps):
        """One compression step of Algorithm 1 on every sampled segment;
        grads(b, e) -> [n, e - b] float32 of this step."""
        self.workers(grads, beta1)
        self.owners_and_updates(lr, eps)
