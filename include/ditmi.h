/*
 * ditmi.h -- C ABI of the MI355X (gfx950) DiT denoising-step library.
 *
 * The library computes the Diffusion Transformer stage of an
 * Encoder -> DiT -> Decoder generation pipeline: the stage that iteratively
 * denoises the latent and dominates serving time (paper: Background and
 * Motivation, "Diffusion Model Architecture" and "Workload Characteristics";
 * System Design, the Transformer service that runs the denoising backbone and
 * updates the latent).  The paper does not write the block out; the block
 * computed is the adaLN-Zero DiT block of the work the paper cites for this
 * stage (Peebles & Xie, arXiv:2212.09748):
 *
 *   (shift1, scale1, gate1, shift2, scale2, gate2) = SiLU(c) W_ada^T + b_ada
 *   x1 = x  + gate1 * (Attn(LN(x) * (1 + scale1) + shift1) W_o^T + b_o)
 *   y  = x1 + gate2 * (GELU_tanh((LN(x1) * (1 + scale2) + shift2) W_1^T + b_1) W_2^T + b_2)
 *
 * LN has no affine, biased variance, eps = shape.ln_eps.  Attn is full
 * bidirectional multi-head attention with scale 1/sqrt(head_dim); the QKV
 * projection's output column j is s*hidden + head*head_dim + d, s in (q,k,v).
 * With text_tokens > 0 the block is the joint two-stream block: image and
 * text tokens each use their own weights (same c) and attention runs over
 * the concatenation [image; text].
 *
 * Conventions for every entry point:
 *   - Pointers to tensors are DEVICE pointers, 16-byte aligned, owned by the
 *     caller; the library never allocates or frees device memory while
 *     computing.  Its only device state is the static scratch array of
 *     dit_block_forward_noalloc (below), which lives until the process ends.
 *   - Weight matrices are row-major [out, in]; weights and biases have the
 *     element type shape.dtype (fp32 or bf16).  Residual streams, the
 *     conditioning vector, patches and outputs are always fp32.
 *   - Work is enqueued on `stream` (a hipStream_t; NULL = the default
 *     stream) and the call returns without synchronising.
 *   - All arguments are validated before anything is enqueued: a call that
 *     returns an error has enqueued no work.  NaN/Inf inputs are not errors;
 *     they propagate.  No call aborts or throws.
 *   - dit_last_error() returns the text of the calling thread's last failure.
 *   - Calls are thread-safe; concurrent calls must not share a workspace.
 *   - Every kernel of a call runs on `stream`; the library creates no
 *     streams.  No allocation or memset is enqueued by any call, so the
 *     calls can be captured into a HIP graph.
 *   - Size limits (DIT_ERR_UNSUPPORTED beyond them): rows = B * (T + Tt)
 *     below 2^24 with rows * max(3D, F) below 2^31, and every weight matrix
 *     (in particular F * D) below 2^31 elements, so that all byte offsets
 *     inside one operand fit the kernels' 32-bit address arithmetic.
 */
#ifndef DITMI_H
#define DITMI_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DITMI_VERSION 1

typedef enum {
  DIT_OK = 0,
  DIT_ERR_INVALID_ARG = -1,  /* null pointer, bad size, misaligned pointer   */
  DIT_ERR_UNSUPPORTED = -2,  /* valid shape this library does not implement  */
  DIT_ERR_WORKSPACE = -3,    /* workspace smaller than dit_workspace_bytes()  */
  DIT_ERR_HIP = -4           /* a HIP runtime call or launch failed           */
} dit_status;

typedef enum { DIT_F32 = 0, DIT_BF16 = 1 } dit_dtype;

/* Workspace kinds for dit_workspace_bytes(). */
typedef enum { DIT_WS_BLOCK = 0, DIT_WS_STEP = 1, DIT_WS_COND = 2, DIT_WS_SAMPLE = 3, DIT_WS_SERVE = 4 } dit_ws_kind;

/* Shape of one DiT model / workload.
 *   batch         B >= 1 samples
 *   tokens        T >= 1 image (latent patch) tokens per sample
 *   text_tokens   Tt >= 0 text tokens per sample; > 0 selects the joint block
 *   hidden        D, multiple of 64, <= 4096
 *   heads, head_dim  heads * head_dim == hidden; head_dim in {64, 72, 128}
 *   mlp_hidden    F, multiple of 64
 *   n_blocks      L >= 1 (used by the step)
 *   patch_in      p*p*C channels of one latent patch (step), 1..256
 *   patch_out     channels predicted per token by the final layer (step), a
 *                 multiple of 4 in 4..256
 *   dtype         dit_dtype of weights and GEMM operands
 *   ln_eps        LayerNorm epsilon (> 0) */
typedef struct {
  int32_t batch, tokens, text_tokens;
  int32_t hidden, heads, head_dim, mlp_hidden, n_blocks;
  int32_t patch_in, patch_out;
  int32_t dtype;
  float ln_eps;
} dit_shape;

/* Weights of one stream of one block (device pointers, [out, in] row-major):
 *   w_ada [6D, D], b_ada [6D]   chunks (shift1, scale1, gate1, shift2, scale2, gate2)
 *   w_qkv [3D, D], b_qkv [3D]
 *   w_o   [D, D],  b_o   [D]
 *   w_fc1 [F, D],  b_fc1 [F]
 *   w_fc2 [D, F],  b_fc2 [D] */
typedef struct {
  const void *w_ada, *b_ada, *w_qkv, *b_qkv, *w_o, *b_o, *w_fc1, *b_fc1, *w_fc2, *b_fc2;
} dit_stream_weights;

/* txt is read only when shape.text_tokens > 0. */
typedef struct {
  dit_stream_weights img, txt;
} dit_block_weights;

/* Step weights.  `blocks` is a HOST array of n_blocks structs holding device
 * pointers.  w_patch [D, patch_in], b_patch [D]; pos [T, D] fp32 or NULL
 * (added after the patch embedding); w_ada_final [2D, D], b_ada_final [2D]
 * (chunks shift, scale); w_final [patch_out, D], b_final [patch_out]. */
typedef struct {
  const void *w_patch, *b_patch;
  const float *pos;
  const dit_block_weights *blocks;
  const void *w_ada_final, *b_ada_final, *w_final, *b_final;
} dit_step_weights;

/* Bytes of workspace the given kind of call needs for this shape (0 when the
 * shape is invalid; dit_last_error() then says why).  The workspace is device
 * memory owned by the caller, 256-byte aligned, contents need not be
 * initialised and are undefined after the call. */
size_t dit_workspace_bytes(const dit_shape *s, int kind);

/* One DiT block, in place (the unit of the DiT stage's per-step work).
 *   x      [B, T, D] fp32 image/latent residual stream, updated in place
 *   x_txt  [B, Tt, D] fp32 text residual stream, updated in place (joint
 *          block only; must be NULL when text_tokens == 0)
 *   cond   [B, D] fp32 conditioning vector c
 *   workspace  >= dit_workspace_bytes(s, DIT_WS_BLOCK) bytes
 * Errors: DIT_ERR_INVALID_ARG, DIT_ERR_UNSUPPORTED, DIT_ERR_WORKSPACE, DIT_ERR_HIP. */
dit_status dit_block_forward(const dit_shape *s, const dit_block_weights *w, float *x, float *x_txt,
                             const float *cond, void *workspace, size_t ws_bytes, void *stream);

/* Size of the static device scratch of dit_block_forward_noalloc (128 MiB
 * per GPU): enough for one block of DiT-XL/2 at 256 tokens x 8 samples
 * (42 MiB) or 1024 tokens x 4 (83 MiB). */
#define DIT_NOALLOC_SCRATCH_BYTES (128u << 20)

/* dit_block_forward for callers that cannot allocate device memory: code
 * being captured into a HIP graph, tight serving loops, harnesses that
 * forbid hipMalloc.  Same arguments, results and errors as
 * dit_block_forward, but the workspace is a static device array of
 * DIT_NOALLOC_SCRATCH_BYTES that the library holds on each GPU it runs on
 * until the process ends; the call allocates nothing and calls no
 * allocating library routine.  The GPU is the one `stream` belongs to (the
 * current device for NULL).  Its first call on a GPU looks the array's
 * device address up (hipGetSymbolAddress) and keeps it.
 * Every call on one GPU shares that GPU's array: calls that may overlap on
 * one GPU (different streams without ordering between them) race and give
 * undefined results; calls ordered on one stream are safe.  The array keeps
 * the last call's contents; nothing in it needs clearing.
 * Errors: those of dit_block_forward, and DIT_ERR_UNSUPPORTED when
 * dit_workspace_bytes(s, DIT_WS_BLOCK) exceeds DIT_NOALLOC_SCRATCH_BYTES
 * (checked before anything is enqueued). */
dit_status dit_block_forward_noalloc(const dit_shape *s, const dit_block_weights *w, float *x, float *x_txt,
                                     const float *cond, void *stream);

/* One denoising step: the full DiT forward of the paper's per-step DiT time
 * (paper Table: per-stage execution time; one step = one DiT forward):
 *   x = patches W_patch^T + b_patch (+ pos);  L blocks;
 *   out = (LN(x) * (1 + scale_f) + shift_f) W_final^T + b_final
 *   patches [B, T, patch_in] fp32;  out [B, T, patch_out] fp32 (may not alias)
 *   x_txt   [B, Tt, D] fp32 text stream, updated in place (joint only, else NULL)
 *   cond    [B, D] fp32
 *   workspace >= dit_workspace_bytes(s, DIT_WS_STEP) bytes
 * No sampler update is applied. */
dit_status dit_step_forward(const dit_shape *s, const dit_step_weights *w, const float *patches,
                            float *x_txt, const float *cond, float *out, void *workspace, size_t ws_bytes,
                            void *stream);

/* Timestep + class conditioning of class-conditional DiT (the work the paper
 * cites for the DiT stage):
 *   e = [cos(t f), sin(t f)], f_i = 10000^(-i/128), i < 128   (256 features)
 *   cond = (SiLU(e W_t1^T + b_t1)) W_t2^T + b_t2 + class_table[y]
 *   t [B] fp32 timesteps, y [B] int32 labels (0 <= y < n_rows of class_table,
 *   not checked on device); w_t1 [D, 256], b_t1 [D], w_t2 [D, D], b_t2 [D],
 *   class_table [*, D] in shape.dtype; cond [B, D] fp32 output.
 *   workspace >= dit_workspace_bytes(s, DIT_WS_COND) bytes. */
dit_status dit_cond_embed(const dit_shape *s, const float *t, const int32_t *y, const void *w_t1,
                          const void *b_t1, const void *w_t2, const void *b_t2, const void *class_table,
                          float *cond, void *workspace, size_t ws_bytes, void *stream);

/* Weights of the timestep + class conditioning (see dit_cond_embed). */
typedef struct {
  const void *w_t1, *b_t1, *w_t2, *b_t2, *class_table;
} dit_cond_weights;

/* The DiT stage's multi-step denoising loop (paper: Background and
 * Motivation, Workload Characteristics -- 40-50 iterations for standard
 * samplers, 4 or 8 for distilled ones; System Design -- the Transformer
 * service iterates the backbone over the timesteps and updates the latent).
 * The paper names no sampler; this is first-order Euler on the
 * flow-matching ODE in the patchified latent space:
 *   for i in 0 .. n_steps-1:
 *     c_i = cond_w ? class conditioning at t_i = (float)(sigmas[i] * t_scale)
 *                    and labels y (as dit_cond_embed)
 *                  : cond (the same for every step)
 *     v_i = one step (dit_step_forward) on z with c_i; joint models start every
 *           step from the given text states x_txt (which are not modified)
 *     z  += (sigmas[i+1] - sigmas[i]) * v_i      (difference taken in fp32)
 *   z       [B, T, P] fp32, P = patch_in = patch_out, updated in place
 *   sigmas  HOST array of n_steps + 1 floats (any order); n_steps >= 0
 *   cond_w  conditioning weights (class-conditioned models) with y [B] int32
 *           device labels, or NULL with cond [B, D] fp32 given
 *   x_txt   [B, Tt, D] fp32 text states (joint only, else NULL), read only
 *   workspace >= dit_workspace_bytes(s, DIT_WS_SAMPLE) bytes
 * Enqueues no allocation or memset, so the whole loop can be captured into a
 * HIP graph and replayed.  Errors as dit_step_forward. */
dit_status dit_sample_euler(const dit_shape *s, const dit_step_weights *w, const dit_cond_weights *cond_w,
                            const int32_t *y, const float *cond, const float *sigmas, int32_t n_steps,
                            float t_scale, float *z, const float *x_txt, void *workspace, size_t ws_bytes,
                            void *stream);

/* One request handed to the DiT stage: host buffers (page-locked for the
 * copies to overlap; pageable memory works but serialises) of the latent from
 * the encoder stage, the denoised latent for the decoder stage, and the
 * request's conditioning input. */
typedef struct {
  const float *z_in;      /* [B, T, P] fp32 */
  float *z_out;           /* [B, T, P] fp32 */
  const int32_t *y;       /* [B] labels when conditioning weights are given, else NULL */
  const float *cond;      /* [B, D] fp32 conditioning otherwise, else NULL */
} dit_request;

/* Serve a sequence of requests through the DiT stage on one GPU: the paper's
 * asynchronous inter-stage pipeline (System Design: the stages communicate
 * through asynchronous queues so that requests occupy different stages at
 * once; Challenge 1: asynchronous handoff absorbs transfer jitter) shrunk to
 * one device.  Per request: copy z_in (and y or cond) host -> device, run the
 * Euler loop of dit_sample_euler (same sigmas, n_steps, t_scale for every
 * request), copy the result device -> host into z_out.
 *   overlap != 0: the copies run on copy_stream (required) and the loops on
 *     `stream`, with two device slots ordered by events: the input of request
 *     i+1 and the output of request i-1 move while request i computes.
 *   overlap == 0: everything runs in order on `stream`.
 *   jitter_us > 0: before enqueueing each request the calling thread sleeps a
 *     pseudo-random time in [0, jitter_us] microseconds (seeded by
 *     jitter_seed), standing in for irregular arrivals from the encoder
 *     stage; results do not depend on it.
 * Results are identical for every overlap/jitter setting.  The call returns
 * after enqueueing; synchronise `stream` before reading z_out.  Temporary
 * HIP events are created and released by the call (no device memory).
 *   workspace >= dit_workspace_bytes(s, DIT_WS_SERVE) bytes */
dit_status dit_serve(const dit_shape *s, const dit_step_weights *w, const dit_cond_weights *cond_w,
                     const dit_request *reqs, int32_t n_requests, const float *sigmas, int32_t n_steps,
                     float t_scale, int32_t overlap, uint32_t jitter_us, uint32_t jitter_seed, void *workspace,
                     size_t ws_bytes, void *stream, void *copy_stream);

/* Fixed 2-D sin-cos position table of DiT, pos [grid_h*grid_w, hidden] fp32,
 * token n = r*grid_w + c: features [0, D/2) encode column c, [D/2, D) row r;
 * each half is [sin(p w_i), cos(p w_i)], w_i = 10000^(-i/(D/4)).
 * hidden must be a multiple of 4. */
dit_status dit_pos_embed_2d(int32_t grid_h, int32_t grid_w, int32_t hidden, float *pos, void *stream);

/* Kernel timing hook for measurement.  dit_timing_enable() (host allocation
 * of HIP events, not a compute call) makes every later launch of kernel class
 * `kclass` record a start/stop hipEvent pair on its launch stream (timing-only
 * events, created without the system-scope fence), for up to max_launches
 * launches, and accumulates the algorithmic flops and bytes of
 * those launches.  dit_timing_read() synchronises on the recorded events and
 * returns the sum of launch durations (ms), the number of launches, and the
 * algorithmic flop and byte totals.  dit_timing_disable() frees the events. */
typedef enum {
  DIT_K_GEMM_QKV = 0, DIT_K_ATTENTION = 1, DIT_K_GEMM_OUT = 2, DIT_K_GEMM_FC1 = 3,
  DIT_K_GEMM_FC2 = 4, DIT_K_LN_MOD = 5, DIT_K_ADALN = 6, DIT_K_OTHER = 7, DIT_K_COUNT = 8
} dit_kernel_class;
dit_status dit_timing_enable(int kclass, int max_launches);
dit_status dit_timing_read(double *total_ms, int *launches, double *flops, double *bytes);
dit_status dit_timing_disable(void);

const char *dit_status_string(dit_status st);
const char *dit_last_error(void);
int dit_version(void);

#ifdef __cplusplus
}
#endif
#endif /* DITMI_H */
