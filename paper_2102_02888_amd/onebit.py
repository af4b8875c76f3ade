"""Python binding of the C ABI in include/onebit.h.

Argument marshalling only: every step of the method runs in the gfx950
kernels of libonebit.so.  Tensors must live on the plan's GPU; float buffers
are torch.float32, sign-bit buffers torch.int64 (the bytes of uint64 words).
Row-major 2-D buffers pass their row stride as the leading dimension.  Calls
are asynchronous on torch's current stream unless a stream is given.
"""
import ctypes

import numpy as np
import torch

from ._native import PlanInfo, call, lib

__all__ = [
    "Plan", "onebit_plan_create", "onebit_warmup_adam_step", "onebit_worker_compress",
    "onebit_server_reduce_compress", "onebit_decompress_update", "onebit_step",
    "onebit_step_noalloc",
    "onebit_error_materialize", "onebit_decode", "onebit_uncompressed_step",
    "onebit_adam_message_step", "onebit_l1_norm", "State",
]


def _stream(stream):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _ptr(t, dtype, name, cols=None, rows=1):
    """Device pointer of a tensor after checking its type, device and layout.
    With `cols`, the tensor must also cover what the kernels touch: `rows`
    rows of `cols` elements (a 1-D tensor is one row), so that a short
    buffer is refused here instead of being read or written out of bounds."""
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch.Tensor" % name)
    if t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if t.device.type != "cuda":
        raise ValueError("%s must be a GPU tensor" % name)
    if t.dim() > 2:
        raise ValueError("%s must be 1-D or 2-D" % name)
    if t.dim() >= 1 and t.stride(-1) != 1:
        raise ValueError("%s must have unit stride in its last dimension" % name)
    if cols is not None:
        have_rows, have_cols = (t.shape[0], t.shape[1]) if t.dim() == 2 else (1, t.numel())
        if have_rows < rows or have_cols < cols:
            raise ValueError("%s is %s; the call needs %d row(s) of at least %d elements"
                             % (name, tuple(t.shape), rows, cols))
    return ctypes.c_void_p(t.data_ptr())


def _flat(t, dtype, name, need):
    """Pointer of a buffer addressed through an explicit leading dimension:
    it must hold at least `need` elements."""
    p = _ptr(t, dtype, name)
    if t.numel() < need:
        raise ValueError("%s has %d elements; the call reads %d" % (name, t.numel(), need))
    return p


_GRAD_DTYPES = {torch.float32: 0, torch.bfloat16: 1, torch.float16: 2}


def _grads(t, cols, rows):
    """(pointer, ONEBIT_GRAD_* code) of a gradient tensor."""
    if not isinstance(t, torch.Tensor) or t.dtype not in _GRAD_DTYPES:
        raise TypeError("grads must be a float32, bfloat16 or float16 tensor")
    return _ptr(t, t.dtype, "grads", cols, rows), _GRAD_DTYPES[t.dtype]


def _ld(t):
    return t.stride(0) if t.dim() == 2 else t.numel()


def _rows(t):
    return t.shape[0] if t.dim() == 2 else 1


def chunk_word_ranges(seg_begin, seg_end, K, n):
    """Per chunk j, the lowest and highest sign word of its segments (k, j)
    over all K tensors (segment q = k*n + j covers elements
    [seg_begin[q], seg_end[q])); -1, -1 for a chunk whose segments are all
    empty.  Computed once per plan, so that a chunk owners' call costs O(n)
    on the host instead of O(K*n)."""
    b = np.asarray(seg_begin, np.int64).reshape(K, n)
    e = np.asarray(seg_end, np.int64).reshape(K, n)
    full = e > b
    big = np.iinfo(np.int64).max
    lo = np.where(full, b // 64, big).min(axis=0)
    hi = np.where(full, (e - 1) // 64, -1).max(axis=0)
    lo[hi < 0] = -1
    return lo, hi


def chunk_extent(chunk_word_lo, chunk_word_hi, K, n, server_begin, server_end):
    """(lowest word, highest word, highest segment) touched by the chunk
    owners [server_begin, server_end), from chunk_word_ranges(); the words are
    -1 if every owned segment is empty."""
    hi = chunk_word_hi[server_begin:server_end]
    lo = chunk_word_lo[server_begin:server_end]
    owned = hi >= 0
    if not owned.any():
        return -1, -1, (K - 1) * n + server_end - 1
    return int(lo[owned].min()), int(hi.max()), (K - 1) * n + server_end - 1


# Modes of Plan.set_server_tables (the ONEBIT_SERVER_TABLES_* constants).
SERVER_TABLES_OFF = 0
SERVER_TABLES_AUTO = 1
SERVER_TABLES_ON = 2


class Plan:
    """Layout of K tensors cut into n chunks, with its device tile tables."""

    def __init__(self, tensor_numel, n_workers):
        numel = np.ascontiguousarray(np.asarray(tensor_numel, dtype=np.int64))
        h = ctypes.c_void_p()
        call("onebit_plan_create", numel.ctypes.data_as(ctypes.c_void_p), len(numel),
             int(n_workers), ctypes.byref(h))
        self._h = h
        info = PlanInfo()
        call("onebit_plan_get_info", h, ctypes.byref(info))
        self.d = info.d
        self.D = info.padded_len
        self.W = info.words
        self.K = info.num_tensors
        self.S = info.num_segments
        self.T = info.num_tiles
        self.n = info.n_workers
        self.tile_elems = info.tile_elems
        self.workspace_bytes = info.workspace_bytes
        self.tensor_off = np.zeros(self.K, np.int64)
        self.seg_begin = np.zeros(self.S, np.int64)
        self.seg_end = np.zeros(self.S, np.int64)
        call("onebit_plan_get_layout", h, self.tensor_off.ctypes.data_as(ctypes.c_void_p),
             self.seg_begin.ctypes.data_as(ctypes.c_void_p),
             self.seg_end.ctypes.data_as(ctypes.c_void_p))
        self.chunk_len = np.zeros(self.K, np.int64)
        call("onebit_plan_info", h, None, None, None,
             self.chunk_len.ctypes.data_as(ctypes.c_void_p), None)
        self.numel = numel
        self.chunk_word_lo, self.chunk_word_hi = chunk_word_ranges(
            self.seg_begin, self.seg_end, self.K, self.n)

    @property
    def workspace_words(self):
        return (self.workspace_bytes + 7) // 8

    def chunk_extent(self, server_begin, server_end):
        """(lowest word, highest word, highest segment) touched by the chunk
        owners [server_begin, server_end); words are -1 if all are empty."""
        return chunk_extent(self.chunk_word_lo, self.chunk_word_hi, self.K, self.n,
                            server_begin, server_end)

    @property
    def handle(self):
        if self._h is None:
            raise ValueError("plan is closed")
        return self._h

    def set_server_tables(self, mode):
        """Where the chunk owners' calls take their lookup tables from:
        SERVER_TABLES_AUTO (the default), SERVER_TABLES_ON (the workspace
        whenever the plan reserved it) or SERVER_TABLES_OFF (built per tile);
        results are identical."""
        call("onebit_plan_set_server_tables", self.handle, int(mode))

    def workspace(self, device):
        nbytes = max(self.workspace_bytes, 256)
        return torch.empty(nbytes // 8 + 32, dtype=torch.float64, device=device)

    def close(self):
        if self._h is not None:
            call("onebit_plan_destroy", self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def onebit_plan_create(tensor_numel, n_workers):
    return Plan(tensor_numel, n_workers)


def onebit_warmup_adam_step(plan, x, m, v, grads, lr, beta1, beta2, eps,
                            bias_correction, step, n_grads=None, stream=None):
    n = _rows(grads) if n_grads is None else n_grads
    if _rows(grads) < n:
        raise ValueError("grads has fewer than %d rows" % n)
    D = plan.D
    call("onebit_warmup_adam_step", plan.handle, _ptr(x, torch.float32, "x", D),
         _ptr(m, torch.float32, "m", D), _ptr(v, torch.float32, "v", D),
         *_grads(grads, D, n), _ld(grads), n, lr, beta1, beta2, eps,
         int(bias_correction), int(step), _stream(stream))


def onebit_worker_compress(plan, m, grads, worker_err, worker_bits, worker_scales, beta1,
                           workspace, n_local=None, m_bits=None, m_scales=None, stream=None):
    """m: fp32 momentum, or None to decode it from (m_bits, m_scales), the
    previous step's gathered server message."""
    n = _rows(grads) if n_local is None else n_local
    if min(_rows(grads), _rows(worker_err), _rows(worker_bits), _rows(worker_scales)) < n:
        raise ValueError("grads, worker_err, worker_bits, worker_scales need %d rows" % n)
    D, W, S = plan.D, plan.W, plan.S
    call("onebit_worker_compress", plan.handle, _ptr(m, torch.float32, "m", D),
         _ptr(m_bits, torch.int64, "m_bits", W), _ptr(m_scales, torch.float32, "m_scales", S),
         *_grads(grads, D, n), _ld(grads), n,
         _ptr(worker_err, torch.float32, "worker_err", D, n), _ld(worker_err),
         _ptr(worker_bits, torch.int64, "worker_bits", W, n), _ld(worker_bits),
         _ptr(worker_scales, torch.float32, "worker_scales", S, n), _ld(worker_scales),
         beta1, _ptr(workspace, torch.float64, "workspace", plan.workspace_words),
         _stream(stream))


def onebit_server_reduce_compress(plan, server_begin, server_end, worker_bits, worker_scales,
                                  server_err, server_bits, server_scales, workspace,
                                  bits_word_base=0, scales_seg_base=0, bits_ld=None,
                                  scales_ld=None, stream=None):
    """Chunk owners [server_begin, server_end).  worker_bits / worker_scales
    are n rows, either the plan-wide arrays (row stride from the tensor) or
    received buffers whose first column is word `bits_word_base` / segment
    `scales_seg_base`, with an explicit row stride bits_ld / scales_ld."""
    n = plan.n
    wlo, whi, qhi = plan.chunk_extent(int(server_begin), int(server_end))
    wcols = whi + 1 - int(bits_word_base) if whi >= 0 else 0
    scols = qhi + 1 - int(scales_seg_base)
    if bits_ld is None:
        bp, bld = _ptr(worker_bits, torch.int64, "worker_bits", wcols, n), _ld(worker_bits)
    else:
        bp, bld = _flat(worker_bits, torch.int64, "worker_bits", (n - 1) * bits_ld + wcols), bits_ld
    if scales_ld is None:
        sp, sld = _ptr(worker_scales, torch.float32, "worker_scales", scols, n), _ld(worker_scales)
    else:
        sp, sld = (_flat(worker_scales, torch.float32, "worker_scales",
                         (n - 1) * scales_ld + scols), scales_ld)
    call("onebit_server_reduce_compress", plan.handle, int(server_begin), int(server_end),
         bp, bld, int(bits_word_base), sp, sld, int(scales_seg_base),
         _ptr(server_err, torch.float32, "server_err", plan.D),
         _ptr(server_bits, torch.int64, "server_bits", plan.W),
         _ptr(server_scales, torch.float32, "server_scales", plan.S),
         _ptr(workspace, torch.float64, "workspace", plan.workspace_words), _stream(stream))


def onebit_decompress_update(plan, server_bits, server_scales, x, m_out, v_frozen, lr, eps,
                             stream=None):
    D = plan.D
    call("onebit_decompress_update", plan.handle,
         _ptr(server_bits, torch.int64, "server_bits", plan.W),
         _ptr(server_scales, torch.float32, "server_scales", plan.S),
         _ptr(x, torch.float32, "x", D), _ptr(m_out, torch.float32, "m_out", D),
         _ptr(v_frozen, torch.float32, "v_frozen", D), lr, eps, _stream(stream))


def _step_args(name, plan, x, m, v_frozen, grads, worker_err, server_err, worker_bits,
               worker_scales, server_bits, server_scales, lr, beta1, eps):
    """The arguments the fused step's entry points share, up to eps."""
    n, D, W, S = plan.n, plan.D, plan.W, plan.S
    # the step addresses worker_bits / worker_scales with row strides W and S
    for t, tname, cols in ((worker_bits, "worker_bits", W), (worker_scales, "worker_scales", S)):
        if t is not None and t.dim() == 2 and cols > 0 and t.stride(0) != cols:
            raise ValueError("%s must be contiguous [n, %d] for %s" % (tname, cols, name))
    return [plan.handle, _ptr(x, torch.float32, "x", D),
            _ptr(m, torch.float32, "m", D), _ptr(v_frozen, torch.float32, "v_frozen", D),
            *_grads(grads, D, n), _ld(grads),
            _ptr(worker_err, torch.float32, "worker_err", D, n), _ld(worker_err),
            _ptr(server_err, torch.float32, "server_err", D),
            _ptr(worker_bits, torch.int64, "worker_bits", W, n),
            _ptr(worker_scales, torch.float32, "worker_scales", S, n),
            _ptr(server_bits, torch.int64, "server_bits", W),
            _ptr(server_scales, torch.float32, "server_scales", S), lr, beta1, eps]


def onebit_step(plan, x, m, v_frozen, grads, worker_err, server_err, worker_bits,
                worker_scales, server_bits, server_scales, lr, beta1, eps, workspace,
                stream=None, events=None):
    """The fused step.  events: optional four torch.cuda.Event objects
    (already recorded once, so that their HIP events exist) marked on the
    stream before the worker pass, the chunk owners' pass and the update, and
    after the update (onebit_step_events)."""
    args = _step_args("onebit_step", plan, x, m, v_frozen, grads, worker_err, server_err,
                      worker_bits, worker_scales, server_bits, server_scales, lr, beta1, eps)
    args.append(_ptr(workspace, torch.float64, "workspace", plan.workspace_words))
    if events is None:
        call("onebit_step", *args, _stream(stream))
        return
    if len(events) != 4:
        raise ValueError("events must hold four torch.cuda.Event objects")
    handles = (ctypes.c_void_p * 4)()
    for k, ev in enumerate(events):
        if ev is not None:
            if not ev.cuda_event:
                raise ValueError("events[%d] has no HIP event yet: record it once first" % k)
            handles[k] = ev.cuda_event
    call("onebit_step_events", *args, handles, _stream(stream))


def onebit_step_noalloc(plan, x, m, v_frozen, grads, worker_err, server_err, worker_bits,
                        worker_scales, server_bits, server_scales, lr, beta1, eps, stream=None):
    """onebit_step without a workspace: the library's static scratch array on
    the device holds the partial sums (calls on one GPU share it and must not
    overlap)."""
    args = _step_args("onebit_step_noalloc", plan, x, m, v_frozen, grads, worker_err,
                      server_err, worker_bits, worker_scales, server_bits, server_scales, lr,
                      beta1, eps)
    call("onebit_step_noalloc", *args, _stream(stream))


def onebit_decode(plan, bits, scales, out, stream=None):
    call("onebit_decode", plan.handle, _ptr(bits, torch.int64, "bits", plan.W),
         _ptr(scales, torch.float32, "scales", plan.S), _ptr(out, torch.float32, "out", plan.D),
         _stream(stream))


def onebit_uncompressed_step(plan, x, m, v_frozen, grads, lr, beta1, eps, n_grads=None,
                             stream=None):
    n = _rows(grads) if n_grads is None else n_grads
    if _rows(grads) < n:
        raise ValueError("grads has fewer than %d rows" % n)
    D = plan.D
    call("onebit_uncompressed_step", plan.handle, _ptr(x, torch.float32, "x", D),
         _ptr(m, torch.float32, "m", D), _ptr(v_frozen, torch.float32, "v_frozen", D),
         *_grads(grads, D, n), _ld(grads), n, lr, beta1, eps, _stream(stream))


def onebit_adam_message_step(plan, x, m, v, bits, scales, lr, beta1, beta2, eps, bias_correction,
                             step, stream=None):
    D = plan.D
    call("onebit_adam_message_step", plan.handle, _ptr(x, torch.float32, "x", D),
         _ptr(m, torch.float32, "m", D), _ptr(v, torch.float32, "v", D),
         _ptr(bits, torch.int64, "bits", plan.W), _ptr(scales, torch.float32, "scales", plan.S),
         lr, beta1, beta2, eps, int(bias_correction), int(step), _stream(stream))


def onebit_l1_norm(plan, v, workspace, out, stream=None):
    """||v||_1 over the real elements into out (a one-element float64 GPU tensor)."""
    call("onebit_l1_norm", plan.handle, _ptr(v, torch.float32, "v", plan.D),
         _ptr(workspace, torch.float64, "workspace", plan.workspace_words),
         _ptr(out, torch.float64, "out", 1), _stream(stream))


def onebit_error_materialize(plan, err_state, scales, delta_out, rows=None, stream=None):
    r = _rows(err_state) if rows is None else rows
    D = plan.D
    call("onebit_error_materialize", plan.handle,
         _ptr(err_state, torch.float32, "err_state", D, r), _ld(err_state),
         _ptr(scales, torch.float32, "scales", plan.S, r), _ld(scales), r,
         _ptr(delta_out, torch.float32, "delta_out", D, r), _ld(delta_out), _stream(stream))


def paired_rows(n, D, grad_dtype, device):
    """(grads, worker_err): [n, D] row views into one zeroed allocation whose
    row i holds worker i's D gradients (grad_dtype) and then its D fp32
    errors.  The two rows that the worker pass streams together then keep one
    fixed offset from each other in memory, where two separate allocations
    land wherever the allocator puts them, and some of those placements run
    the pass up to 5% slower.  D must be a positive multiple of 64 (a plan's
    padded length), which keeps every row 16-byte aligned."""
    if D <= 0 or D % 64:
        raise ValueError("D must be a positive multiple of 64, got %d" % D)
    gsize = torch.empty((), dtype=grad_dtype).element_size()
    pair = torch.zeros((n, (gsize + 4) * D), dtype=torch.uint8, device=device)
    return pair[:, :gsize * D].view(grad_dtype), pair[:, gsize * D:].view(torch.float32)


class State:
    """Device buffers of one compression-stage run with n_local simulated
    workers (all zero-initialised except x, m, v which the caller fills).

    With packed_momentum (the default) every compression step after the first
    takes the momentum from the previous step's server message instead of
    the fp32 buffer `m`, which then goes stale; momentum() returns the
    current value either way."""

    def __init__(self, plan, device, n_local=None, grad_rows=None, packed_momentum=True,
                 grad_dtype=torch.float32, grads=None):
        """grads: an existing [rows, >= D] gradient tensor to read (shared,
        not copied) instead of a new zero one."""
        n = plan.n if n_local is None else n_local
        D, W, S = plan.D, plan.W, plan.S
        f = dict(dtype=torch.float32, device=device)
        self.plan = plan
        self.n_local = n
        self.x = torch.zeros(D, **f)
        self.m = torch.zeros(D, **f)
        self.v = torch.zeros(D, **f)
        if grads is None and grad_rows in (None, n) and D > 0:
            self.grads, self.worker_err = paired_rows(n, D, grad_dtype, device)
        else:
            if grads is None:
                grads = torch.zeros((n if grad_rows is None else grad_rows, D), dtype=grad_dtype,
                                    device=device)
            self.grads = grads
            self.worker_err = torch.zeros((n, D), **f)
        self.worker_bits = torch.zeros((n, W), dtype=torch.int64, device=device)
        self.worker_scales = torch.zeros((n, S), **f)
        self.server_err = torch.zeros(D, **f)
        self.server_bits = torch.zeros(W, dtype=torch.int64, device=device)
        self.server_scales = torch.zeros(S, **f)
        self.workspace = plan.workspace(device)
        self.packed_momentum = packed_momentum
        self.compression_steps = 0

    # Everything a later step reads: parameters, moments, both error states
    # with the scales that complete them, and the last server message (the
    # packed momentum).  Gradients and worker sign words are per-step outputs.
    STATE_KEYS = ("x", "m", "v", "worker_err", "worker_scales", "server_err", "server_bits",
                  "server_scales")

    def state_dict(self):
        """Host copies of the state (CPU tensors; safetensors can store them)."""
        out = {k: getattr(self, k).detach().cpu().clone() for k in self.STATE_KEYS}
        out["compression_steps"] = torch.tensor([self.compression_steps], dtype=torch.int64)
        out["packed_momentum"] = torch.tensor([int(self.packed_momentum)], dtype=torch.int64)
        return out

    def load_state_dict(self, sd):
        """Restores a state_dict() into this state's device buffers (same plan
        shape); the next step continues bit for bit."""
        for k in self.STATE_KEYS:
            dst = getattr(self, k)
            src = sd[k]
            if tuple(src.shape) != tuple(dst.shape) or src.dtype != dst.dtype:
                raise ValueError("%s: expected %s %s, got %s %s" % (
                    k, tuple(dst.shape), dst.dtype, tuple(src.shape), src.dtype))
            dst.copy_(src)
        self.compression_steps = int(sd["compression_steps"][0])
        self.packed_momentum = bool(int(sd["packed_momentum"][0]))

    def warmup(self, lr, beta1, beta2, eps, step, bias_correction=0, stream=None):
        onebit_warmup_adam_step(self.plan, self.x, self.m, self.v, self.grads, lr, beta1,
                                beta2, eps, bias_correction, step, stream=stream)

    def momentum_is_packed(self):
        return self.packed_momentum and self.compression_steps > 0

    def step(self, lr, beta1, eps, stream=None, events=None):
        """One compression step (onebit_step); events: see onebit_step."""
        m = None if self.momentum_is_packed() else self.m
        onebit_step(self.plan, self.x, m, self.v, self.grads, self.worker_err,
                    self.server_err, self.worker_bits, self.worker_scales, self.server_bits,
                    self.server_scales, lr, beta1, eps, self.workspace, stream=stream,
                    events=events)
        self.compression_steps += 1

    def step_uncompressed(self, lr, beta1, eps, stream=None):
        """One step of the "1-bit Adam (32-bits)" comparison variant (fp32 m)."""
        onebit_uncompressed_step(self.plan, self.x, self.m, self.v, self.grads, lr, beta1, eps,
                                 stream=stream)

    def step_naive(self, lr, beta1, beta2, eps, t, stream=None):
        """One step of the "Adam(1-bit Naive)" comparison variant: the gradient
        is error-compensated and compressed by every worker (the worker pass
        with beta1 = 0 over a zero momentum), averaged and recompressed by the
        chunk owners, and Adam updates m and v from the decoded result."""
        if not hasattr(self, "_plus_bits"):
            # With beta1 = 0 the worker's momentum term is 0 * m.  Decoded from
            # all-ones sign words and zero scales, m is +0 everywhere, and
            # 0 * +0 is the same +0 that a zero fp32 momentum gives, so the
            # packed-momentum pass computes exactly what the fp32-momentum
            # row walk would, reading 1/8 byte of m per element and row.
            self._plus_bits = torch.full((self.plan.W,), -1, dtype=torch.int64,
                                         device=self.x.device)
            self._zero_scales = torch.zeros(self.plan.S, dtype=torch.float32,
                                            device=self.x.device)
        onebit_worker_compress(self.plan, None, self.grads, self.worker_err,
                               self.worker_bits, self.worker_scales, 0.0, self.workspace,
                               n_local=self.n_local, m_bits=self._plus_bits,
                               m_scales=self._zero_scales, stream=stream)
        onebit_server_reduce_compress(self.plan, 0, self.plan.n, self.worker_bits,
                                      self.worker_scales, self.server_err, self.server_bits,
                                      self.server_scales, self.workspace, stream=stream)
        onebit_adam_message_step(self.plan, self.x, self.m, self.v, self.server_bits,
                                 self.server_scales, lr, beta1, beta2, eps, 0, t, stream=stream)

    def variance_l1_norm(self, stream=None):
        """||v||_1 (fp64) computed on the GPU; synchronises to return it."""
        if not hasattr(self, "_norm"):
            self._norm = torch.zeros(1, dtype=torch.float64, device=self.v.device)
        onebit_l1_norm(self.plan, self.v, self.workspace, self._norm, stream=stream)
        if stream is not None:
            stream.synchronize()
        return float(self._norm.item())

    def momentum(self):
        if self.compression_steps > 1 and self.packed_momentum:
            out = torch.zeros_like(self.m)
            onebit_decode(self.plan, self.server_bits, self.server_scales, out)
            return out
        return self.m

    def worker_delta(self):
        out = torch.zeros_like(self.worker_err)
        onebit_error_materialize(self.plan, self.worker_err, self.worker_scales, out)
        return out

    def server_delta(self):
        out = torch.zeros_like(self.server_err)
        onebit_error_materialize(self.plan, self.server_err, self.server_scales, out, rows=1)
        return out
