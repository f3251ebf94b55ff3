"""MI355X (gfx950) encoder-stage library: the forward and backward pass of a
contiguous block of post-LN BERT encoder layers on one GPU, in hand-written
HIP kernels behind a C ABI (include/stage.h)."""
from .binding import (PARAM_NAMES, SAVED_NAMES, STAGE_BF16, STAGE_F32, Stage, StageError,
                      load_library, stage_backward, stage_destroy, stage_forward, stage_grad,
                      stage_init, stage_last_error, stage_param, stage_read, stage_set_param,
                      stage_set_stream, stage_site_count, stage_site_name,
                      stage_tensor_bytes, stage_trace_mask, stage_trace_read,
                      stage_trace_site)

__all__ = ["Stage", "StageError", "load_library", "PARAM_NAMES", "SAVED_NAMES", "STAGE_BF16",
           "STAGE_F32", "stage_init", "stage_set_stream", "stage_forward", "stage_backward",
           "stage_param", "stage_grad", "stage_set_param", "stage_read", "stage_tensor_bytes",
           "stage_last_error", "stage_destroy", "stage_trace_site", "stage_trace_mask", "stage_trace_read",
           "stage_site_count", "stage_site_name"]
