"""MI355X (gfx950) encoder-stage library: the forward and backward pass of a
contiguous block of post-LN BERT encoder layers on one GPU, in hand-written
HIP kernels behind a C ABI (include/stage.h), and the host-side layer
allocator that sizes such blocks per device (include/alloc.h)."""
from .binding import (ALLOC_CT_PER_DEVICE, ALLOC_CT_PER_LAYER, ALLOC_EINVAL, ALLOC_ENOFIT,
                      ALLOC_OK, PARAM_NAMES, SAVED_NAMES, STAGE_BF16, STAGE_F32, AllocError,
                      Stage, StageError, alloc_coarse, alloc_fine, alloc_workloads, load_library,
                      stage_backward, stage_backward_noalloc, stage_destroy, stage_device_bytes, stage_forward, stage_grad, stage_init,
                      stage_init_units, stage_memory_model_units,
                      stage_last_error, stage_memory_model, stage_mfma_peak, stage_param, stage_read, stage_record_grads,
                      stage_set_param,
                      stage_set_stream, stage_site_count, stage_site_name, stage_tensor_bytes,
                      stage_trace_mask, stage_trace_read, stage_trace_site)

__all__ = ["Stage", "StageError", "load_library", "PARAM_NAMES", "SAVED_NAMES", "STAGE_BF16",
           "STAGE_F32", "stage_init", "stage_init_units", "stage_memory_model_units", "stage_set_stream", "stage_forward", "stage_backward",
           "stage_backward_noalloc",
           "stage_param", "stage_grad", "stage_set_param", "stage_read", "stage_tensor_bytes",
           "stage_last_error", "stage_destroy", "stage_trace_site", "stage_trace_mask", "stage_trace_read",
           "stage_site_count", "stage_site_name", "stage_device_bytes", "stage_memory_model",
           "stage_mfma_peak", "stage_record_grads",
           "AllocError", "ALLOC_OK", "ALLOC_EINVAL", "ALLOC_ENOFIT", "ALLOC_CT_PER_LAYER",
           "ALLOC_CT_PER_DEVICE", "alloc_coarse", "alloc_fine", "alloc_workloads"]
