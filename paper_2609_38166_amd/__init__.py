"""LeapQuant 8-bit recurrent-state decode path for MI355X (gfx950).

The compute path is the HIP library ``libleapquant.so`` behind the C ABI in
``include/leapquant.h``; :mod:`.binding` passes torch device tensors to it.
:mod:`.synth` draws the seeded synthetic workloads.
"""
from . import binding  # noqa: F401  (loads the library lazily, on first call)
from .binding import (  # noqa: F401
    LeapQuantError, State, lq_dims, make_dims, leapquant_state_bytes, leapquant_quantize_state,
    leapquant_decode_step, leapquant_decode_step_general, leapquant_decode_step_commit,
    leapquant_window_commit,
    leapquant_baseline_step, leapquant_baseline_step_general, leapquant_dequantize_state,
    leapquant_check_error,
)

__all__ = [
    "LeapQuantError", "State", "lq_dims", "make_dims", "leapquant_state_bytes",
    "leapquant_quantize_state", "leapquant_decode_step", "leapquant_decode_step_general",
    "leapquant_decode_step_commit", "leapquant_window_commit", "leapquant_baseline_step", "leapquant_baseline_step_general",
    "leapquant_dequantize_state", "leapquant_check_error",
]
