/*
 * pulse_tstage.h -- C ABI of the skip-collocated stage for transformer-block
 * denoisers (UViT family) on MI355X (gfx950).
 *
 * The method applies to every UNet-like denoiser whose long skips join an
 * encoder block to a decoder block, the transformer-block models included
 * (Sec. II-A; evaluated on UViT and Hunyuan-DiT, Sec. VII).  As for the
 * ResBlock stage (pulse_stage.h), a device holds an encoder group whose block
 * outputs are kept as skips in local memory and the decoder group that
 * consumes them (symmetric placement, Sec. IV-B; stage pairing, Sec. V-B);
 * the backward pass splits the decoder input gradient and buffers the skip
 * gradient locally until the encoder's backward adds it (Sec. I; Sec. III).
 *
 * Block arithmetic (the paper leaves it open; pre-norm UViT block):
 *   h = x + Proj(MHA(LN1(x))),  y = h + Fc2(GELU(Fc1(LN2(h))))
 * LayerNorm over each token's channels (biased variance, eps inside the
 * square root, affine g/b); MHA with head dimension 64, q k^T scaled by
 * 1/8 and a row softmax, heads splitting the channels in order and q, k, v
 * stacked in that order along the qkv projection's output; GELU in the erf
 * form; an MLP of mlp_ratio * width hidden channels; every linear layer has a
 * bias.  Decoder block k first applies Skip_k, a linear layer width -> width
 * over the token-wise concatenation [v || skip] (upstream channels first);
 * the concatenation is never materialised: the skip linear's GEMMs read
 * both sources in place.  Encoder block k caches its output in skip slot k;
 * decoder block k reads slot n_enc - 1 - k (mirror order).
 *
 * Conventions (as in pulse_stage.h): tensor pointers are caller-owned
 * DEVICE memory valid until the enqueued work has run; activations are
 * token-major [batch, tokens, width] bf16, contiguous, 16-byte aligned;
 * parameters and gradients are fp32.  Nothing here allocates device memory:
 * the caller binds one workspace of pulse_tstage_sizes() bytes.  Every call
 * validates before it enqueues anything; on error it returns a status !=
 * PULSE_OK, changes no state and pulse_last_error() says why.  A stage is
 * not thread-safe, and every call on one handle shares its scratch
 * buffers: enqueue them on one stream, or order the streams yourself.
 */
#ifndef PULSE_TSTAGE_H
#define PULSE_TSTAGE_H

#include "pulse_stage.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct pulse_tstage pulse_tstage; /* opaque, library-owned */

typedef struct {
  int32_t batch;        /* images per microbatch                              */
  int32_t tokens;       /* tokens per image: a multiple of 64, at most 4096    */
  int32_t width;        /* channels C = 64 * heads, at most 2048               */
  int32_t heads;        /* attention heads of dimension 64                     */
  int32_t mlp_ratio;    /* MLP hidden width = mlp_ratio * width (1..8)         */
  float eps;            /* LayerNorm epsilon (>= 0)                            */
  pulse_dtype dtype;    /* activation dtype: PULSE_BF16 only                   */
  int32_t n_enc;        /* encoder blocks (>= 1)                               */
  int32_t n_dec;        /* decoder blocks: must equal n_enc                    */
  int32_t max_inflight; /* microbatches that may coexist (1..64)               */
  uint32_t flags;       /* PULSE_FLAG_DRY_RUN: bookkeeping only                */
} pulse_tstage_desc;

/* Validate and create.  PULSE_E_SHAPE when a rule above fails or the token
 * count batch * tokens exceeds 2^20. */
pulse_status pulse_tstage_create(const pulse_tstage_desc* desc, pulse_tstage** out);
void pulse_tstage_destroy(pulse_tstage* st);

/* Number of fp32 parameters (and gradients) and the workspace bytes; either
 * pointer may be NULL. */
pulse_status pulse_tstage_sizes(const pulse_tstage* st, int64_t* n_params,
                                size_t* workspace_bytes);

/* Flat fp32 parameter layout, in order: for each encoder block k the tensors
 * "enc{k}.NAME", NAME in ln1.g ln1.b qkv.W qkv.b proj.W proj.b ln2.g ln2.b
 * fc1.W fc1.b fc2.W fc2.b; then for each decoder block k "dec{k}.skip.W"
 * [C, 2C], "dec{k}.skip.b" and the same twelve.  Linear weights are [out,
 * in]: qkv.W [3C, C], proj.W [C, C], fc1.W [rC, C], fc2.W [C, rC].  `name`
 * receives the NUL-terminated name, `offset` the element offset, `shape` up
 * to 4 extents (unused = 0).  idx = -1 writes the tensor count to *offset. */
pulse_status pulse_tstage_param_layout(const pulse_tstage* st, int32_t idx, char name[64],
                                       int64_t* offset, int32_t shape[4]);

/* Bind fp32 params and grads (n_params each; grads ACCUMULATE) and the
 * workspace (256-byte aligned, at least workspace_bytes). */
pulse_status pulse_tstage_bind(pulse_tstage* st, const float* params, float* grads,
                               void* workspace, size_t workspace_bytes);

/* Refresh the bf16 weight copies (the forward [out][in] layout and the
 * transposed [in][out] layout of the data-gradient GEMMs) from the fp32
 * params.  Call after bind and after every parameter update. */
pulse_status pulse_tstage_sync_params(pulse_tstage* st, void* stream);

/* Forward of one half for microbatch `mb` (any id >= 0).
 *  ENC: in = x, out = y_enc; fills every skip slot of mb.
 *  DEC: in = u, out = y_dec; reads the skip slots of mb.
 * Both [batch, tokens, width] bf16.  Order per microbatch: ENC fwd, DEC fwd,
 * DEC bwd, ENC bwd; PULSE_E_STATE otherwise, PULSE_E_CACHE_FULL beyond
 * max_inflight microbatches. */
pulse_status pulse_tstage_forward(pulse_tstage* st, pulse_half half, int32_t mb,
                                  const void* in, void* out, void* stream);

/* Backward of one half for microbatch `mb`.
 *  DEC: dout = dL/dy_dec, din = dL/du; buffers the gradient of every skip
 *       slot read (fp32, in the workspace).
 *  ENC: dout = dL/dy_enc, din = dL/dx; adds each slot's buffered gradient
 *       to the gradient reaching that encoder output, then releases mb.
 * Parameter gradients are ACCUMULATED (+=). */
pulse_status pulse_tstage_backward(pulse_tstage* st, pulse_half half, int32_t mb,
                                   const void* dout, void* din, void* stream);

/* Overlapped decoder backward (default off), as pulse_stage_overlap_bwd: a
 * DEC backward returns without waiting for its last parameter-gradient work
 * on the stage's second stream; an ENC backward of the same microbatch on
 * the same stream starts beside it, and any other call (or
 * pulse_tstage_flush on a stream) orders that work before what follows it.
 * The decoder half's parameter gradients are complete in `stream` order only
 * after that.  Results are bitwise those of the switch off. */
pulse_status pulse_tstage_overlap_bwd(pulse_tstage* st, int32_t enable);

/* Work enqueued on `stream` after this call is ordered after the stage's
 * side-stream work, including what an overlapped decoder backward left
 * running.  Enqueues only stream waits. */
pulse_status pulse_tstage_flush(pulse_tstage* st, void* stream);

/* Copy the buffered gradient of (mb, slot) (fp32 [batch, tokens, width])
 * into dst without consuming it: an inspection hook for tests.
 * PULSE_E_CACHE_MISS when absent. */
pulse_status pulse_tstage_skip_grad(const pulse_tstage* st, int32_t mb, int32_t slot,
                                    float* dst, void* stream);

pulse_status pulse_tstage_release(pulse_tstage* st, int32_t mb);
pulse_status pulse_tstage_reset(pulse_tstage* st);
int32_t pulse_tstage_inflight(const pulse_tstage* st);

/* Per-kernel timing of the GEMM launches (the implicit-GEMM kernel in its
 * token-major 1x1 form): each is bracketed by HIP events on the call's
 * stream.  _read synchronises them and returns the launch count, summed ms,
 * summed FLOPs (2 M N K) and summed compulsory bytes since the last reset;
 * any output pointer may be NULL. */
pulse_status pulse_tstage_timing(pulse_tstage* st, int32_t enable);
pulse_status pulse_tstage_timing_read(pulse_tstage* st, int64_t* launches, double* ms,
                                      double* flops, double* bytes);

/* Execute steps [t0, t1) of device d's row of a collocated wave schedule
 * (Sec. V; the table format of pulse_sched_build) on a transformer stage:
 * each cell becomes pulse_tstage_forward/backward of the ENC half (stage
 * s = d forward, s = 4D-1-d backward) or DEC half (s = 2D-1-d forward,
 * s = 2D+d backward) for that microbatch, in step order, on `stream`.  The
 * boundary tensors come from io[m] (x, u, g_enc, g_dec in; y_enc, y_dec, dx,
 * du out; temb and dtemb are not used).  PULSE_E_INVALID_ARG when
 * 0 <= t0 <= t1 <= T fails or a cell in the range is not one of the
 * device's four stages (nothing is enqueued then); otherwise the first
 * failing stage call's status. */
pulse_status pulse_tsched_run_device(pulse_tstage* st, int32_t D, int32_t d, int32_t M,
                                     const int32_t* table, int32_t T, int32_t t0, int32_t t1,
                                     const pulse_mb_io* io, void* stream);

/* FLOPs of one microbatch's ENC+DEC forward and backward: 2 M N K over every
 * linear-layer GEMM (forward, data and weight gradient) plus the attention
 * products (q k^T and p v forward; d p, d q, d k and d v backward). */
double pulse_tstage_flops(const pulse_tstage* st);

#ifdef __cplusplus
}
#endif

#endif /* PULSE_TSTAGE_H */
