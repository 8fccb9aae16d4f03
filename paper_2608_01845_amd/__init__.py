"""MI355X-native WorldDynCache denoising rollout (gfx950 HIP kernels behind a C ABI).

The library ``libwdc.so`` (include/wdc.h) holds every kernel and the rollout
control; this package is its ctypes binding. Build it with
``python -m paper_2608_01845_amd.build``.
"""
from ._binding import (  # noqa: F401
    MODE_ALL_EXACT, MODE_FORCED, MODE_PERIODIC, MODE_RISK, OBS_KERNEL, OBS_LINEAR, POST_EXACT, POST_SURROGATE,
    PRE_DECISION, SURROGATE_LIFTED, SURROGATE_SECANT, TIMING_CLASSES, Context, ModelDesc, Params, State, StepLog,
    WdcError, default_params, desc_from_config, exported_symbols, load,
)
