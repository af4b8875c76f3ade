"""1-bit Adam's compression-stage hot path on AMD MI355X (gfx950).

The kernels and their C ABI live in ``libonebit.so`` (sources in ``csrc/``,
header ``include/onebit.h``); this package is the Python binding.
"""
from .onebit import (  # noqa: F401
    Plan, State, SERVER_TABLES_AUTO, SERVER_TABLES_OFF, SERVER_TABLES_ON, onebit_decode, onebit_decompress_update, onebit_error_materialize,
    onebit_plan_create,
    onebit_server_reduce_compress, onebit_step, onebit_step_noalloc, onebit_warmup_adam_step,
    onebit_worker_compress, onebit_uncompressed_step, onebit_adam_message_step, onebit_l1_norm,
)
from .freeze import VarianceFreezeDetector  # noqa: F401
from .optimizer import OnebitAdam  # noqa: F401
from ._native import OnebitError, lib  # noqa: F401
