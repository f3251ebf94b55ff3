/*
 * stage.h - C ABI of the MI355X (gfx950) encoder-stage library.
 *
 * A "stage" is a contiguous block of L post-LN BERT encoder layers that the
 * layer allocator places on one device (paper section III: each device
 * turns the previous device's output tensor into its own output, and after
 * the forward pass computes its layers' gradients in reverse order).  One
 * encoder layer (section II-C) is self-attention per Eq. (1),
 * softmax(Q K^T / sqrt(d_k)) V with Q, K, V the input times three matrices,
 * followed by three linear layers with residual connections: h -> h, h -> f
 * (widening) and f -> h.  A LayerNorm follows each residual addition and the
 * widening layer is followed by the exact erf GELU.
 *
 * Conventions
 *   - Activations x, y, dy, dx are row-major [batch, seq, hidden] in the
 *     stage dtype (fp32 or bf16), on the device, owned by the caller.
 *   - key_mask is uint8 [batch, seq] on the device, owned by the caller;
 *     1 = the key position may be attended, 0 = padding.  NULL = no padding.
 *   - Parameters (per layer, in stage_param_id order) are owned by the
 *     library: matrices in the stage dtype, row-major [out, in]; biases,
 *     LayerNorm gammas and betas in fp32.  W_qkv stacks the query, key and
 *     value matrices as row blocks [0,h), [h,2h), [2h,3h); head j owns
 *     columns [64 j, 64 j + 64) of each projection.
 *   - Gradients are fp32, owned by the library, overwritten (not
 *     accumulated) by every stage_backward.
 *   - All device work is enqueued on the stage's HIP stream; calls return
 *     without synchronising unless stated.  Results are valid once the
 *     caller has synchronised that stream.
 *   - Every call returns a stage_status; nothing aborts or throws across
 *     the ABI.  stage_last_error gives a message for the last failure.
 */
#ifndef SKY_STAGE_H
#define SKY_STAGE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Enumerations are int-sized on both sides of the ABI.  Compiled as C++
 * they get a fixed underlying type int, so that every int a C caller passes
 * is a value of the type there too (and is rejected by the argument checks
 * when it is not one of the listed values), instead of being undefined. */
#ifndef SKY_ENUM_INT
#ifdef __cplusplus
#define SKY_ENUM_INT : int
#else
#define SKY_ENUM_INT
#endif
#endif

typedef struct stage stage_t; /* opaque, library-owned */

typedef enum SKY_ENUM_INT {
  STAGE_OK = 0,
  STAGE_EINVAL = 1, /* invalid argument: dims, null pointer, index range */
  STAGE_ESTATE = 2, /* call out of order, e.g. backward without forward */
  STAGE_ENOMEM = 3, /* device allocation failed */
  STAGE_EHIP = 4    /* a HIP runtime call or kernel launch failed */
} stage_status;

typedef enum SKY_ENUM_INT { STAGE_F32 = 0, STAGE_BF16 = 1 } stage_dtype;

typedef enum SKY_ENUM_INT {
  STAGE_W_QKV = 0, /* [3h, h]  dtype */
  STAGE_B_QKV = 1, /* [3h]     fp32  */
  STAGE_W_O = 2,   /* [h, h]   dtype */
  STAGE_B_O = 3,   /* [h]      fp32  */
  STAGE_G1 = 4,    /* [h]      fp32, LayerNorm after attention */
  STAGE_BE1 = 5,   /* [h]      fp32  */
  STAGE_W_1 = 6,   /* [f, h]   dtype */
  STAGE_B_1 = 7,   /* [f]      fp32  */
  STAGE_W_2 = 8,   /* [h, f]   dtype */
  STAGE_B_2 = 9,   /* [h]      fp32  */
  STAGE_G2 = 10,   /* [h]      fp32, LayerNorm after the FFN */
  STAGE_BE2 = 11,  /* [h]      fp32  */
  STAGE_NPARAM = 12
} stage_param_id;

/* Saved activations of the latest forward pass (for layer-wise checks). */
typedef enum SKY_ENUM_INT {
  STAGE_SAVED_X = 0,   /* layer input           [T, h]  dtype */
  STAGE_SAVED_QKV = 1, /* Q | K | V             [T, 3h] dtype */
  STAGE_SAVED_CTX = 2, /* attention context     [T, h]  dtype */
  STAGE_SAVED_H1 = 3,  /* first LayerNorm out   [T, h]  dtype */
  STAGE_SAVED_GD = 4,  /* GELU'(U), U = FFN pre-activation [T, f] dtype */
  STAGE_SAVED_G = 5,   /* GELU(U)               [T, f]  dtype */
  STAGE_NSAVED = 6
} stage_saved_id;

/*
 * Create a stage of L_stage layers (sections II-C and III).
 *   hidden: h, a multiple of 64, at most 2048;  heads: h / heads must be 64;
 *   ffn: f, a multiple of 64.  seed: weights are drawn N(0, 0.02) by a
 *   counter-based generator (splitmix64 of seed, layer, tensor and index,
 *   Box-Muller) and rounded to dtype; biases and betas 0, gammas 1.
 *   hip_stream: hipStream_t the stage enqueues on (NULL = default stream).
 * On success *out owns device memory for parameters and gradients; release
 * it with stage_destroy.  EINVAL on bad dims, ENOMEM / EHIP on failure (then
 * *out is NULL).
 */
stage_status stage_init(int L_stage, int hidden, int heads, int ffn, uint64_t seed,
                        stage_dtype dtype, void* hip_stream, stage_t** out);

/*
 * Create a stage that starts and ends at half-layer boundaries.  The layer
 * allocator of section IV places discrete layers, whose count may exceed
 * the number of encoder layers (the strong-scaling model of section VI-G
 * counts several allocation units per encoder layer).  Here every encoder
 * layer is two units, cut where a single tensor crosses in each direction:
 *   unit 2j     attention half of layer j: QKV projection, attention, output
 *               projection, residual add and first LayerNorm (X -> H1);
 *   unit 2j + 1 feed-forward half of layer j: widening layer and GELU,
 *               narrowing layer, residual add and second LayerNorm
 *               (H1 -> Y; H1 is also the residual).
 * The stage holds units [first_unit, first_unit + n_units): its layer l is
 * global layer first_unit / 2 + l, and L_stage = (last unit) / 2 -
 * first_unit / 2 + 1 layers are indexed in stage_param, stage_grad,
 * stage_read, ...  Its input is X of its first unit's layer (H1 when
 * first_unit is odd) and its output is that of its last unit.  Chaining the
 * stages of a partition of [0, 2 L) computes the same function as one stage
 * of L layers, except that on bf16 stages the tensors that cross a stage
 * boundary are rounded to bf16 there (they are the stage's input and output
 * in its dtype): an H1 that crosses a boundary reaches the second LayerNorm
 * rounded (inside a stage it is added with its rounding residual, to about
 * 16 significant bits), and in the backward pass the
 * gradient that crosses a boundary is rounded (inside a stage the residual
 * stream of the backward pass stays in fp32).  Weights are drawn as in stage_init with the global
 * layer index, so a layer has the same weights in every stage that holds
 * it; stage_init(L, ...) is stage_init_units(0, 2 L, ...).  Parameters,
 * gradients and saved tensors of the absent half of a partial layer do not
 * exist: stage_param, stage_grad, stage_set_param and stage_read return
 * EINVAL for them (saved X, QKV, CTX belong to the attention half; H1, GD,
 * G to the feed-forward half) and stage_tensor_bytes returns 0.
 * EINVAL for first_unit < 0, n_units < 1, first_unit + n_units > 2^30 or
 * dims stage_init rejects; otherwise as stage_init.
 */
stage_status stage_init_units(int first_unit, int n_units, int hidden, int heads, int ffn,
                              uint64_t seed, stage_dtype dtype, void* hip_stream, stage_t** out);

/* Change the stream later calls enqueue on. */
stage_status stage_set_stream(stage_t* s, void* hip_stream);

/*
 * Forward pass of the stage (section III): y = layer_{L-1}(...layer_0(x)).
 * x, y: [batch, seq, h] device, stage dtype; x and y may not alias.
 * key_mask: [batch, seq] uint8 device or NULL.  batch, seq >= 0 (an empty
 * batch is valid).  x and key_mask are copied into the saved context, so
 * the caller may reuse them once the stream has passed this call.  The
 * saved context replaces any earlier one.  (Activation buffers are
 * (re)allocated when the token count grows.)
 */
stage_status stage_forward(stage_t* s, const void* x, const uint8_t* key_mask, int batch,
                           int seq, void* y);

/*
 * Backward pass (section III: gradients in reverse layer order) of
 * <y, dy> for the latest forward.  dy, dx: [batch, seq, h] device, stage
 * dtype.  Writes dx and overwrites all parameter gradients.  Consumes the
 * saved context: a second call without a new forward returns ESTATE.
 */
stage_status stage_backward(stage_t* s, const void* dy, void* dx);

/*
 * For callers that cannot allocate device memory during the call (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * stage_backward with the same kernels and results, bitwise, whose
 * weight-gradient split-K partials and bias / LayerNorm column partial sums
 * live in a static device array of 256 MiB (one per device, held from the
 * library's first use on that device until the process ends) instead of
 * buffers of the stage.  It calls no allocator (no hipMalloc / hipFree, no
 * HIP events: stage tracing does not see its launches).  Every call on a
 * device shares that device's array and leaves its contents behind: calls
 * that overlap on one device (several stages on concurrent streams) race
 * and must be serialised by the caller.  EINVAL (context kept) when the
 * batch needs more partial results than the array holds: the split-K
 * partials grow with h f (about 201 MB at most for h = 1024, f = 4096, and
 * for h = 2048, f = 8192), the column partial sums with the token count
 * (about 2.6 KB per token at h = 2048); e.g. h = 2048, f = 8192 at 32768
 * tokens does not fit.  Otherwise as stage_backward.
 */
stage_status stage_backward_noalloc(stage_t* s, const void* dy, void* dx);

/*
 * Device memory.  stage_device_bytes: bytes the library holds for s
 * (parameters, gradients, the saved-activation record and the workspace, as
 * requested from hipMalloc).  stage_memory_model: the same figure predicted
 * without a device for a stage of these dims after a forward of batch x seq
 * tokens, split into per_layer (one layer's parameters, gradients and saved
 * activations: the layer memory lm that the allocator's benchmark stage
 * measures, section IV-B) and shared (workspace held once per stage), so
 * that a stage of L layers holds L * per_layer + shared.  EINVAL for dims
 * stage_init rejects or negative batch / seq.  Host arithmetic only.
 */
stage_status stage_device_bytes(const stage_t* s, int64_t* bytes);
stage_status stage_memory_model(int hidden, int heads, int ffn, int batch, int seq,
                                stage_dtype dtype, int64_t* per_layer, int64_t* shared);
/*
 * The same per allocation unit (see stage_init_units): a stage of units
 * [u0, u0 + n) holds shared + (its attention units) * attn_unit + (its
 * feed-forward units) * ffn_unit bytes, and per_layer = attn_unit +
 * ffn_unit.  The attention unit counts X, QKV, the score or log-sum-exp
 * record, the context and the first LayerNorm's saved rows; the
 * feed-forward unit counts its input H1, GELU'(U), G and the second
 * LayerNorm's saved rows; each counts its own parameters and gradients.
 */
stage_status stage_memory_model_units(int hidden, int heads, int ffn, int batch, int seq,
                                      stage_dtype dtype, int64_t* attn_unit, int64_t* ffn_unit,
                                      int64_t* shared);

/*
 * Device pointer, element count and dtype of parameter `which` of `layer`.
 * Section III: each device holds the weights of its own layers for the
 * whole of training (fetched once at the start) and updates them locally;
 * the pointer stays valid until stage_destroy, so the caller's optimiser can
 * update the weights in place between steps.  EINVAL for an index out of
 * range or a half-layer the stage does not hold.
 */
stage_status stage_param(stage_t* s, int layer, int which, void** dev_ptr, int64_t* numel,
                         stage_dtype* dtype);

/*
 * Device pointer (fp32) and element count of that parameter's gradient.
 * Section III: after its backward pass a device uses the gradients of its
 * own layers to update their weights locally; they are never sent to
 * another device.  Overwritten by every stage_backward; valid until
 * stage_destroy.  Errors as stage_param.
 */
stage_status stage_grad(stage_t* s, int layer, int which, float** dev_ptr, int64_t* numel);

/*
 * Copy `bytes` bytes from src (host or device) into parameter `which` of
 * `layer` (bytes must equal numel * element size of its dtype).
 * Synchronises the stage stream before returning.
 */
stage_status stage_set_param(stage_t* s, int layer, int which, const void* src, size_t bytes);

/*
 * Copy a library-owned tensor into dst (host or device), synchronously on
 * the stage stream.  kind 0 = parameter, 1 = gradient, 2 = saved activation
 * (stage_saved_id; needs a saved context), 3 = the gradient that reached
 * layer `layer`'s output in the latest backward (which = 0; fp32 [T, h];
 * needs stage_record_grads, else ESTATE).  bytes must equal the tensor's
 * size in bytes (fp32 for gradients).
 */
stage_status stage_read(stage_t* s, int kind, int layer, int which, void* dst, size_t bytes);

/*
 * Record, in every later backward, the gradient that reaches each layer's
 * output (section III: the gradients flow through the layers in reverse
 * order; on bf16 stages this is the fp32 residual stream inside the stage),
 * for layer-wise checks through stage_read kind 3.  on = 1 or 0.  Takes
 * effect at the next stage_forward, which (re)allocates T * h * 4 bytes per
 * layer for the record (or frees it); the current saved context is
 * dropped.  EINVAL for other values of on.
 */
stage_status stage_record_grads(stage_t* s, int on);

/* Bytes of the tensor stage_read(kind, layer, which) would copy (0 if none). */
size_t stage_tensor_bytes(stage_t* s, int kind, int layer, int which);

/*
 * Tracing (the paper times forward and backward work per module to profile
 * devices, section V-B).  stage_trace_site(s, site) makes every later launch
 * of kernel site `site` (0 <= site < stage_site_count(); -1 = off) record a
 * pair of HIP events on the stage stream around it, and clears earlier
 * records.  stage_trace_read synchronises the stream and returns how many
 * traced launches ran and their summed event time in ms, then clears the
 * records.  Tracing adds two event records per traced launch and nothing
 * to untraced ones.
 */
stage_status stage_trace_site(stage_t* s, int site);
/* Same for a set of sites: bit i of mask selects site i (0 = off). */
stage_status stage_trace_mask(stage_t* s, uint64_t mask);
stage_status stage_trace_read(stage_t* s, int* launches, double* total_ms);
int stage_site_count(void);
const char* stage_site_name(int site); /* "" for an unknown site */

/*
 * Achievable dense bf16 MFMA throughput of the current device and the mean
 * shader clock it held meanwhile: one work-group per compute unit, each
 * wavefront issuing independent chains of 32x32x16 bf16 MFMAs on register
 * operands for `iters` iterations (no memory traffic), timed with HIP events
 * on hip_stream (NULL = default stream); the clock is the shader-cycle
 * counter over the constant-rate counter.  Synchronous.  Writes TFLOP/s and
 * GHz; EINVAL for null outputs or iters outside [1, 2^24], EHIP if the run
 * fails.  Allocates and frees a few bytes of device memory per call.
 */
stage_status stage_mfma_peak(void* hip_stream, int iters, double* tflops, double* clock_ghz);

/* Message describing the last failure on this handle ("" if none); with
 * s == NULL, the message of the last failed stage_init on this thread. */
const char* stage_last_error(const stage_t* s);

/* Free everything the handle owns (synchronises its stream). NULL is a no-op. */
void stage_destroy(stage_t* s);

#ifdef __cplusplus
}
#endif
#endif /* SKY_STAGE_H */
