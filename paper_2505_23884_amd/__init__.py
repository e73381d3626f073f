"""MI355X (gfx950) LaCT fast-weight layer forward and its backward.

Thin ctypes binding over ``liblact.so`` (see ``include/lact.h``): it only
marshals torch tensors into device pointers, picks the current HIP stream and
allocates the workspace. Every step of the path runs in the library's HIP
kernels; there is no CPU or PyTorch fallback.
"""
from .binding import (  # noqa: F401
    LactError, LactDesc, lib, load_library, workspace_bytes, forward, forward_noalloc, forward_momentum,
    forward_schedule, forward_linear, backward, backward_linear, backward_workspace_bytes, backward_momentum,
    backward_momentum_workspace_bytes, backward_schedule, prologue, rmsnorm_out,
    prologue_backward, rmsnorm_out_backward, check_desc,
    timing_enable, timing_reset, timing_read, KCLASS_NAMES,
    APPLY_THEN_UPDATE, UPDATE_THEN_APPLY, IO_BF16, IO_FP32, SEG_MODES, FW_SWIGLU, FW_LINEAR,
)
