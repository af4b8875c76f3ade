"""ctypes loader for libonebit.so (the gfx950 kernels and their C ABI).

There is no fallback: if the library has not been built the import of the
binding fails loudly.  Build it with ``python -m paper_2102_02888_amd.build``
(or ``__graft_entry__.build()``).
"""
import ctypes
import os

from .build import LIB as LIB_PATH

_vp = ctypes.c_void_p
_i64 = ctypes.c_int64
_i32 = ctypes.c_int32
_f32 = ctypes.c_float


class PlanInfo(ctypes.Structure):
    _fields_ = [("d", ctypes.c_int64), ("padded_len", ctypes.c_int64),
                ("words", ctypes.c_int64), ("num_tensors", ctypes.c_int64),
                ("num_segments", ctypes.c_int64), ("num_tiles", ctypes.c_int64),
                ("n_workers", ctypes.c_int32), ("tile_elems", ctypes.c_int32),
                ("workspace_bytes", ctypes.c_size_t)]


# name -> argtypes (every function returns int32 status unless listed below)
SIGNATURES = {
    "onebit_plan_create": [_vp, _i32, _i32, _vp],
    "onebit_plan_destroy": [_vp],
    "onebit_plan_get_info": [_vp, _vp],
    "onebit_plan_set_server_tables": [_vp, _i32],
    "onebit_plan_get_layout": [_vp, _vp, _vp, _vp],
    "onebit_plan_info": [_vp, _vp, _vp, _vp, _vp, _vp],
    "onebit_warmup_adam_step": [_vp, _vp, _vp, _vp, _vp, _i32, _i64, _i32, _f32, _f32, _f32,
                                _f32, _i32, _i64, _vp],
    "onebit_worker_compress": [_vp, _vp, _vp, _vp, _vp, _i32, _i64, _i32, _vp, _i64, _vp, _i64,
                               _vp, _i64, _f32, _vp, _vp],
    "onebit_server_reduce_compress": [_vp, _i32, _i32, _vp, _i64, _i64, _vp, _i64, _i64, _vp,
                                      _vp, _vp, _vp, _vp],
    "onebit_decompress_update": [_vp, _vp, _vp, _vp, _vp, _vp, _f32, _f32, _vp],
    "onebit_step": [_vp, _vp, _vp, _vp, _vp, _i32, _i64, _vp, _i64, _vp, _vp, _vp, _vp, _vp,
                    _f32, _f32, _f32, _vp, _vp],
    "onebit_step_noalloc": [_vp, _vp, _vp, _vp, _vp, _i32, _i64, _vp, _i64, _vp, _vp, _vp, _vp,
                            _vp, _f32, _f32, _f32, _vp],
    "onebit_step_events": [_vp, _vp, _vp, _vp, _vp, _i32, _i64, _vp, _i64, _vp, _vp, _vp, _vp,
                           _vp, _f32, _f32, _f32, _vp, _vp, _vp],
    "onebit_decode": [_vp, _vp, _vp, _vp, _vp],
    "onebit_l1_norm": [_vp, _vp, _vp, _vp, _vp],
    "onebit_uncompressed_step": [_vp, _vp, _vp, _vp, _vp, _i32, _i64, _i32, _f32, _f32, _f32,
                                 _vp],
    "onebit_adam_message_step": [_vp, _vp, _vp, _vp, _vp, _vp, _f32, _f32, _f32, _f32, _i32,
                                 _i64, _vp],
    "onebit_error_materialize": [_vp, _vp, _i64, _vp, _i64, _i32, _vp, _i64, _vp],
    "onebit_status_str": [_i32],
    "onebit_last_error": [],
}
RESTYPES = {"onebit_status_str": ctypes.c_char_p, "onebit_last_error": ctypes.c_char_p}

_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(
                "libonebit.so is not built (%s); run `python -m paper_2102_02888_amd.build`"
                % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        for name, args in SIGNATURES.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = RESTYPES.get(name, ctypes.c_int32)
        _lib = L
    return _lib


class OnebitError(RuntimeError):
    def __init__(self, func, status):
        L = lib()
        self.status = status
        super().__init__("%s: %s: %s" % (func, L.onebit_status_str(status).decode(),
                                         L.onebit_last_error().decode()))


def call(name, *args):
    st = getattr(lib(), name)(*args)
    if st != 0:
        raise OnebitError(name, st)
    return st
