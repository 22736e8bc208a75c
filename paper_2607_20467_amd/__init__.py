"""MI355X (gfx950) implementation of one DC-Leap denoising iteration.

The work happens in ``libdcl.so`` (hand-written HIP kernels behind a C ABI, declared in
``include/dcl.h``); ``binding`` marshals arguments to it with ctypes and PyTorch supplies device
memory and streams. There is no CPU fallback: loading fails loudly when the library is missing.
"""
from .binding import (  # noqa: F401
    DCL_DTYPE_BF16, DCL_DTYPE_F32, DCL_SCORE_ALL_UNCOMMITTED, DCL_SCORE_SUPPRESS_MASK, DCL_SEL_CONTIGUOUS_DRAFTS,
    DCL_SEL_MARGIN, DCL_SEL_NO_PROGRESS_GUARD, DCL_SEL_NONCONTIGUOUS, DCL_SEL_SCORE_ALL,
    DclError, DclLayerTaps, Runner, config_from_geometry, dcl_debug_gemm_plan, dcl_debug_layer, dcl_debug_logits,
    dcl_denoise_step, dcl_generate, dcl_kv_append,
    dcl_last_error, dcl_load_weights, dcl_model_create, dcl_model_destroy, dcl_profile_enable, dcl_profile_read,
    dcl_score_hidden, dcl_score_workspace_bytes, dcl_select_contiguous, dcl_status_string, dcl_weights_bytes,
    dcl_workspace_bytes, library_path, load_library,
)
from . import binding  # noqa: F401,E402
from .binding import DCL_NOALLOC_SCRATCH_BYTES, dcl_denoise_step_noalloc  # noqa: F401,E402
