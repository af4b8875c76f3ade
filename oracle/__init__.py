"""CPU oracle of the 1-bit Adam hot path -- TEST INFRASTRUCTURE ONLY.

A thin numpy/ctypes wrapper over ``onebit_oracle.c``.  Only ``tests/``,
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may use
it; the GPU library never does, and the two share no code.

Every function works on numpy arrays in the flat padded layout documented in
``onebit_oracle.c`` (tensor offsets rounded up to 64 elements, chunk length
64*ceil(d/(64 n)), LSB-first sign bits in uint64 words, bit 1 <=> value >= 0).
"""
import ctypes
import os

import numpy as np

from . import build as _build

_lib = None

_f32p = np.ctypeslib.ndpointer(dtype=np.float32, flags="C_CONTIGUOUS")
_i64p = np.ctypeslib.ndpointer(dtype=np.int64, flags="C_CONTIGUOUS")
_u64p = np.ctypeslib.ndpointer(dtype=np.uint64, flags="C_CONTIGUOUS")
_vp = ctypes.c_void_p
_i64 = ctypes.c_int64
_i32 = ctypes.c_int32
_f32 = ctypes.c_float


def lib():
    """Loads the oracle library, building it first if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        L = ctypes.CDLL(_build.LIB)
        L.orc_chunk_len.restype = _i64
        L.orc_chunk_len.argtypes = [_i64, _i32]
        L.orc_layout.restype = _i64
        L.orc_layout.argtypes = [_i64p, _i32, _i32, _i64p, _i64p, _i64p]
        L.orc_compress.restype = _f32
        L.orc_compress.argtypes = [_i64, _i64, _f32p, _u64p]
        L.orc_decode.restype = _f32
        L.orc_decode.argtypes = [_u64p, _i64, _f32]
        L.orc_l1_norm_range.restype = ctypes.c_double
        L.orc_l1_norm_range.argtypes = [_i64, _i64, _vp]
        L.orc_decode_range.restype = None
        L.orc_decode_range.argtypes = [_i64, _i64, _vp, _f32, _vp]
        L.orc_warmup_range.restype = None
        L.orc_warmup_range.argtypes = [_i64, _i64, _vp, _vp, _vp, _vp, _i64, _i32,
                                       _f32, _f32, _f32, _f32, _i32, _i64]
        L.orc_worker_segment.restype = _f32
        L.orc_worker_segment.argtypes = [_i64, _i64, _f32, _vp, _vp, _vp, _vp, _vp]
        L.orc_server_segment.restype = _f32
        L.orc_server_segment.argtypes = [_i64, _i64, _i32, _vp, _i64, _vp, _i64,
                                         _vp, _vp, _vp]
        L.orc_update_segment.restype = None
        L.orc_update_segment.argtypes = [_i64, _i64, _vp, _f32, _f32, _f32, _vp, _vp, _vp]
        L.orc_step.restype = None
        L.orc_step.argtypes = [_i64p, _i32, _i32, _i64p, _i64p,
                               _vp, _vp, _vp, _vp, _i64, _vp, _i64,
                               _vp, _vp, _i64, _vp, _vp, _vp,
                               _f32, _f32, _f32, _vp]
        L.orc_step_uncompressed_range.restype = None
        L.orc_step_uncompressed_range.argtypes = [_i64, _i64, _i32, _vp, _vp, _vp,
                                                  _vp, _i64, _f32, _f32, _f32]
        _lib = L
    return _lib


def _ptr(a, dtype):
    assert isinstance(a, np.ndarray) and a.dtype == dtype and a.flags.c_contiguous, \
        (type(a), getattr(a, "dtype", None))
    return a.ctypes.data


def _f(a):
    return _ptr(a, np.float32)


def _u(a):
    return _ptr(a, np.uint64)


class Layout:
    """Tensor offsets, padded length and (tensor, chunk) segments."""

    def __init__(self, numel, n):
        self.numel = np.ascontiguousarray(np.asarray(numel, dtype=np.int64))
        self.K = len(self.numel)
        self.n = int(n)
        self.S = self.K * self.n
        self.tensor_off = np.zeros(self.K, np.int64)
        self.seg_begin = np.zeros(self.S, np.int64)
        self.seg_end = np.zeros(self.S, np.int64)
        self.D = int(lib().orc_layout(self.numel, self.K, self.n, self.tensor_off,
                                      self.seg_begin, self.seg_end))
        self.W = self.D // 64

    def chunk_len(self, k):
        return int(lib().orc_chunk_len(int(self.numel[k]), self.n))

    def segments(self):
        return list(zip(self.seg_begin.tolist(), self.seg_end.tolist()))

    def real_mask(self):
        """Boolean [D] mask of real (non-padding) elements."""
        mask = np.zeros(self.D, bool)
        for off, d in zip(self.tensor_off.tolist(), self.numel.tolist()):
            mask[off:off + d] = True
        return mask


def compress(z, b=0, e=None):
    """C[z] on z[b:e]: returns (bits uint64[ceil(len(z)/64)], scale)."""
    z = np.ascontiguousarray(z, dtype=np.float32)
    e = len(z) if e is None else e
    bits = np.zeros((len(z) + 63) // 64, np.uint64)
    s = lib().orc_compress(b, e, z, bits)
    return bits, np.float32(s)


def decode(bits, e, scale):
    return np.float32(lib().orc_decode(bits, int(e), float(scale)))


def l1_norm(layout, v):
    """||v||_1 over the real elements of the layout (binary64, tensor order)."""
    total = 0.0
    for off, d in zip(layout.tensor_off.tolist(), layout.numel.tolist()):
        total += lib().orc_l1_norm_range(off, off + d, _f(v))
    return total


def decode_message(layout, bits, scales):
    """Decoded message over the padded layout: +-scale of each element's
    segment (padding 0)."""
    out = np.zeros(layout.D, np.float32)
    for q, (b, e) in enumerate(layout.segments()):
        lib().orc_decode_range(b, e, _u(bits), float(scales[q]), _f(out))
    return out


def warmup_step(layout, x, m, v, g, n_grads, lr, beta1, beta2, eps,
                bias_correction, t):
    """One warm-up Adam step on every real element (in place on x, m, v).
    g has n_grads rows of equal stride."""
    g = np.ascontiguousarray(g)
    g_ld = g.shape[-1] if g.ndim == 2 else len(g)
    L = lib()
    for off, d in zip(layout.tensor_off.tolist(), layout.numel.tolist()):
        if d > 0:
            L.orc_warmup_range(off, off + d, _f(x), _f(m), _f(v), _f(g), g_ld,
                               int(n_grads), lr, beta1, beta2, eps,
                               int(bias_correction), int(t))


def warmup_range(b, e, x, m, v, g, g_ld, n_grads, lr, beta1, beta2, eps, bias_correction, t):
    """Warm-up step on elements [b, e) of flat arrays; g: n_grads rows of g_ld."""
    lib().orc_warmup_range(int(b), int(e), _f(x), _f(m), _f(v), _f(g), int(g_ld), int(n_grads),
                           lr, beta1, beta2, eps, int(bias_correction), int(t))


def worker_segment(b, e, beta1, m, g_i, delta_i, bits_i, z_scratch):
    return np.float32(lib().orc_worker_segment(b, e, beta1, _f(m), _f(g_i), _f(delta_i),
                                               _u(bits_i), _f(z_scratch)))


def server_segment(b, e, n, wbits, bits_ld, wscale, scale_stride, delta_bar,
                   bits_out, z_scratch):
    """wbits: flat uint64 array of n rows of stride bits_ld, addressed by global
    word index; wscale: flat float32 array whose element i*scale_stride is
    worker i's scale for this segment."""
    return np.float32(lib().orc_server_segment(b, e, int(n), _u(wbits), int(bits_ld),
                                               _f(wscale), int(scale_stride),
                                               _f(delta_bar), _u(bits_out),
                                               _f(z_scratch)))


def update_segment(b, e, bits, scale, lr, eps, x, m, v_frozen):
    lib().orc_update_segment(b, e, _u(bits), float(scale), lr, eps, _f(x),
                             None if m is None else _f(m), _f(v_frozen))


class State:
    """Full compression-stage state of n simulated workers on the host."""

    def __init__(self, layout, x, m, v_frozen):
        L = layout
        self.layout = L
        self.x = np.array(x, np.float32)
        self.m = np.array(m, np.float32)
        self.v = np.array(v_frozen, np.float32)
        self.delta = np.zeros((L.n, L.D), np.float32)
        self.delta_bar = np.zeros(L.D, np.float32)
        self.wbits = np.zeros((L.n, L.W), np.uint64)
        self.wscales = np.zeros((L.n, L.S), np.float32)
        self.sbits = np.zeros(L.W, np.uint64)
        self.sscales = np.zeros(L.S, np.float32)
        self._z = np.zeros(L.D, np.float32)

    def step(self, g, lr, beta1, eps):
        """One compression-stage step; g is [n, D] float32."""
        L = self.layout
        g = np.ascontiguousarray(g, np.float32)
        assert g.shape == (L.n, L.D)
        lib().orc_step(L.numel, L.K, L.n, L.seg_begin, L.seg_end,
                       _f(self.x), _f(self.m), _f(self.v), _f(g), L.D,
                       _f(self.delta), L.D, _f(self.delta_bar),
                       _u(self.wbits), L.W, _f(self.wscales),
                       _u(self.sbits), _f(self.sscales), lr, beta1, eps, _f(self._z))


def step_uncompressed(layout, x, m, v_frozen, g, lr, beta1, eps):
    """One step of the identity-compressor variant on every real element."""
    g = np.ascontiguousarray(g, np.float32)
    L = lib()
    for off, d in zip(layout.tensor_off.tolist(), layout.numel.tolist()):
        if d > 0:
            L.orc_step_uncompressed_range(off, off + d, layout.n, _f(x), _f(m),
                                          _f(v_frozen), _f(g), g.shape[1],
                                          lr, beta1, eps)
