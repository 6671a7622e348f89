/*
 * pulse_stage.h -- C ABI of the MI355X (gfx950) library that runs the
 * per-device compute of one skip-collocated Pulse pipeline stage.
 *
 * The method (Pulse, arXiv 2606.19163) places every encoder block of a UNet
 * denoiser on the same device as the decoder block its long skip connection
 * feeds (symmetric placement: an op in partition q forces its skip partner
 * into partition p-q+1, Sec. IV-B), so with S = 2D stages each device holds
 * encoder stage q and decoder stage 2D-1-q (Sec. V-B).  Skip activations are
 * stored in local buffers during the forward pass and reused in the backward
 * pass, and their gradients are buffered locally as well (Sec. I; Sec. III,
 * Overview).  One `pulse_stage` is that device's share: a group of encoder
 * ResBlocks whose outputs are cached as skips in HBM and a group of decoder
 * ResBlocks that read [upstream || skip] without materialising the
 * concatenation, plus the backward pass that splits the decoder's input
 * gradient and adds the skip gradient into the encoder's backward.
 *
 * Block arithmetic (the paper leaves it open): GroupNorm -> SiLU -> 3x3 conv
 * (+ Linear(SiLU(temb)) broadcast over H x W) -> GroupNorm -> SiLU -> 3x3
 * conv, plus a residual that is the identity when C_in == C_out and a 1x1
 * conv otherwise.  Convs are stride 1; 3x3 convs pad with zeros applied to
 * the conv input after GroupNorm+SiLU.  GroupNorm uses the biased variance
 * with eps inside the square root; in a decoder block its groups follow the
 * concatenated channel index and may hold channels of both sources.
 *
 * Conventions
 *  - Every tensor pointer is caller-owned DEVICE memory that stays valid
 *    until the work enqueued on `stream` has finished.  Activations are NHWC,
 *    contiguous, 16-byte aligned, in the stage dtype (fp32 or bf16) unless
 *    stated otherwise.  Parameters, gradients and dtemb are fp32.
 *  - Nothing here allocates device memory: the caller binds one workspace of
 *    pulse_stage_sizes() bytes for the stage's lifetime.
 *  - Every call validates before it enqueues anything.  On error it returns
 *    a status != PULSE_OK, changes no state, enqueues nothing, and
 *    pulse_last_error() describes the cause.  No exception crosses the ABI.
 *    Kernel faults are asynchronous and surface at the caller's next
 *    synchronisation.
 *  - A stage is not thread-safe: serialise calls on one handle.  Calls may
 *    use different streams: every call shares the stage's scratch buffers,
 *    so a call on a stream other than the previous call's first makes its
 *    stream wait for the previous call's work (an event recorded at the end
 *    of every call that enqueues work).
 *  - Forward and backward calls may be captured into a HIP graph (stream
 *    capture): replays do the captured work with bitwise the eager results.
 *    A replay does not run the host-side bookkeeping, so capture a sequence
 *    that leaves every microbatch where it found it (for example the
 *    forward and backward of both halves of one microbatch).
 */
#ifndef PULSE_STAGE_H
#define PULSE_STAGE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct pulse_stage pulse_stage; /* opaque, library-owned */

typedef enum {
  PULSE_OK = 0,
  PULSE_E_INVALID_ARG = 1,   /* null pointer, bad enum, bad alignment      */
  PULSE_E_SHAPE = 2,         /* descriptor not supported / inconsistent    */
  PULSE_E_STATE = 3,         /* call out of the per-microbatch order       */
  PULSE_E_CACHE_FULL = 4,    /* more than max_inflight microbatches        */
  PULSE_E_CACHE_MISS = 5,    /* skip entry absent                          */
  PULSE_E_CACHE_OCCUPIED = 6,/* skip entry already present                 */
  PULSE_E_NOT_BOUND = 7,     /* no workspace / parameters bound            */
  PULSE_E_HIP = 8            /* a HIP runtime call failed                  */
} pulse_status;

typedef enum { PULSE_F32 = 0, PULSE_BF16 = 1 } pulse_dtype;
typedef enum { PULSE_ENC = 0, PULSE_DEC = 1 } pulse_half;
typedef enum { PULSE_SKIP_ACT = 0, PULSE_SKIP_GRAD = 1 } pulse_skip_kind;

/* skip-entry state bits returned by pulse_skip_cache_state */
#define PULSE_SKIP_ACT_PRESENT 1
#define PULSE_SKIP_GRAD_PRESENT 2

/* stage flags */
#define PULSE_FLAG_DRY_RUN 1u /* validate and run the bookkeeping only: no
                                 workspace, no device work (host tests)   */

/* Encoder ResBlock c_in -> c_out.  skip_slot_out >= 0 caches its output in
 * that skip slot; -1 leaves it uncached. */
typedef struct {
  int32_t c_in, c_out, skip_slot_out;
} pulse_enc_block;

/* Decoder ResBlock reading [upstream (c_up) || skip (c_skip)] -> c_out; the
 * skip comes from slot skip_slot_in.  c_up + c_skip != c_out, so its
 * residual is always a 1x1 conv. */
typedef struct {
  int32_t c_up, c_skip, c_out, skip_slot_in;
} pulse_dec_block;

typedef struct {
  int32_t batch, height, width; /* per microbatch                          */
  int32_t groups;               /* GroupNorm groups (divides every C)      */
  float eps;                    /* GroupNorm epsilon                        */
  int32_t temb_dim;             /* timestep-embedding width                 */
  pulse_dtype dtype;            /* activation storage dtype                 */
  int32_t n_enc;
  const pulse_enc_block* enc;   /* encoder blocks in forward order          */
  int32_t n_dec;
  const pulse_dec_block* dec;   /* decoder blocks in forward order          */
  int32_t input_skip_slot;      /* >= 0: the stage input is cached there    */
  int32_t max_inflight;         /* microbatches that may coexist (>= 1)     */
  uint32_t flags;               /* PULSE_FLAG_*                             */
} pulse_stage_desc;

/* Validate `desc` and create a stage.  Shape rules (PULSE_E_SHAPE):
 * n_enc, n_dec >= 1; every channel count a multiple of 32 and divisible by
 * `groups`; enc[k].c_in == enc[k-1].c_out; dec[k].c_up == dec[k-1].c_out;
 * every slot is filled by exactly one producer (an encoder block or the
 * stage input), read by at most one decoder block, and the reader's c_skip
 * equals the producer's channel count; slots are in [0, 64).
 * *out receives the handle; free it with pulse_stage_destroy. */
pulse_status pulse_stage_create(const pulse_stage_desc* desc, pulse_stage** out);
void pulse_stage_destroy(pulse_stage* st);

/* Number of fp32 parameters (the same count holds the gradients) and the
 * workspace size in bytes.  Either out pointer may be NULL. */
pulse_status pulse_stage_sizes(const pulse_stage* st, int64_t* n_params,
                               size_t* workspace_bytes);

/* Flat fp32 parameter layout.  Tensor `idx` (0 <= idx < count) is named
 * "enc{k}.NAME" / "dec{k}.NAME" with NAME one of W1 b1 Wl bl g1 be1 g2 be2
 * W2 b2 Ws bs; W1/W2 are OHWI [O,3,3,I], Ws is [O,I], Wl is [O,temb_dim].
 * `name` receives a NUL-terminated string (< 64 bytes), `offset` the element
 * offset in the flat buffer, `shape` up to 4 extents (unused = 0).  Passing
 * idx = -1 writes the tensor count into *offset. */
pulse_status pulse_stage_param_layout(const pulse_stage* st, int32_t idx,
                                      char name[64], int64_t* offset,
                                      int32_t shape[4]);

/* Bind caller memory: `params` and `grads` are fp32 device buffers of
 * n_params elements laid out as above (grads ACCUMULATE: the caller zeroes
 * them per iteration); `workspace` is a device buffer of at least
 * workspace_bytes, 256-byte aligned.  Must precede sync/forward/backward. */
pulse_status pulse_stage_bind(pulse_stage* st, const float* params, float* grads,
                              void* workspace, size_t workspace_bytes);

/* Refresh the library's compute copies of the weights (stage-dtype shadows,
 * the flipped/transposed data-gradient layouts and folded biases) from the
 * fp32 master params.  Call after bind and after every parameter update. */
pulse_status pulse_stage_sync_params(pulse_stage* st, void* stream);

/* Forward of one half for microbatch `mb` (any id >= 0).
 *  ENC: in = x [B,H,W,enc[0].c_in], out = y_enc [B,H,W,enc[last].c_out].
 *       Fills the skip slots of every caching block (and input_skip_slot).
 *  DEC: in = u [B,H,W,dec[0].c_up], out = y_dec [B,H,W,dec[last].c_out].
 *       Reads skip slot dec[k].skip_slot_in of `mb` for every block k.
 *  temb = [B, temb_dim] in the stage dtype.  The stage keeps copies of what
 *  its backward needs, so `in` and `temb` may be reused once the enqueued
 *  work has run.  Order per microbatch: ENC fwd (or pulse_skip_cache_put of
 *  every slot the decoder reads), DEC fwd, DEC bwd, ENC bwd. */
pulse_status pulse_stage_forward(pulse_stage* st, pulse_half half, int32_t mb,
                                 const void* in, const void* temb, void* out,
                                 void* stream);

/* For callers that cannot allocate device memory per call or allocate at
 * all (code under HIP graph capture, tight serving loops, harnesses that
 * forbid it): pulse_stage_forward with the forward pass's scratch (GroupNorm
 * partial sums, timestep projections, conv K-split partials) taken from a
 * device array of PULSE_FWD_STATIC_SCRATCH_BYTES that the library holds on
 * each GPU it runs on until the process ends, instead of from the bound
 * workspace.  Same arguments, semantics and results as pulse_stage_forward
 * (bitwise); it makes no allocation of its own.  PULSE_E_SHAPE when the
 * stage's forward scratch exceeds the array (the 64x64x320 stage at batch 8
 * needs about 5.3 MB; stages with K-split convs or wide channels at large
 * batch do not fit); PULSE_E_STATE while per-launch timing is on.  Every
 * call on one GPU shares that GPU's array: calls that may overlap on one
 * GPU (any stage, any stream) race and must be serialised by the caller.
 * The array is written before it is read in every call, so it needs no
 * clearing. */
#define PULSE_FWD_STATIC_SCRATCH_BYTES (8u << 20)
pulse_status pulse_stage_forward_static(pulse_stage* st, pulse_half half, int32_t mb,
                                        const void* in, const void* temb, void* out,
                                        void* stream);

/* Backward of one half for microbatch `mb`.
 *  DEC: dout = dL/dy_dec, din = dL/du.  Writes the skip-gradient entry of
 *       every slot the decoder reads.
 *  ENC: dout = dL/dy_enc, din = dL/dx.  Adds the buffered skip gradient of
 *       every cached block output (and of the cached stage input), then
 *       releases the microbatch.
 *  dout/din are in the stage dtype.  Parameter gradients and
 *  dtemb_accum ([B, temb_dim], fp32, may be NULL) are ACCUMULATED (+=). */
pulse_status pulse_stage_backward(pulse_stage* st, pulse_half half, int32_t mb,
                                  const void* dout, void* din, float* dtemb_accum,
                                  void* stream);

/* Overlapped decoder backward (default off).  The backward pass runs the
 * parameter gradients (weight GEMMs, bias and timestep sums) on a second
 * stream of the stage beside the data-gradient chain, and every backward
 * call normally ends by making `stream` wait for that stream.  With this
 * switch on, a DEC backward returns without that wait: the parameter-
 * gradient work of its last block may still run, and an ENC backward of the
 * same microbatch on the same stream starts beside it (it waits only where
 * it writes a buffer that work still reads).  That work is ordered before
 * everything enqueued on a stream after the next call on the stage (which
 * joins it), or after pulse_stage_flush on that stream.  So with the switch
 * on, the decoder half's parameter gradients and its dtemb_accum
 * contributions are complete in `stream` order only after the next call or
 * a flush (a device-wide synchronisation also covers them).  The results
 * are bitwise those of the switch off.  It saves the wait where a
 * microbatch's encoder backward follows its decoder backward on the device
 * (a stage holding two adjacent pipeline stages, as the device with the
 * two middle stages of a skip-collocated pipeline does). */
pulse_status pulse_stage_overlap_bwd(pulse_stage* st, int32_t enable);

/* Work enqueued on `stream` after this call is ordered after all work the
 * stage has enqueued, on any stream, including parameter-gradient work an
 * overlapped decoder backward left running.  Enqueues only stream waits. */
pulse_status pulse_stage_flush(pulse_stage* st, void* stream);

/* Copy `src` ([B,H,W,C_slot], stage dtype) into the activation entry of
 * (mb, slot) and mark it present: the hook by which a skip produced on
 * another device enters the cache (partial collocation, Sec. VIII-B).
 * PULSE_E_CACHE_OCCUPIED if present, PULSE_E_CACHE_FULL if `mb` would need
 * a row beyond max_inflight. */
pulse_status pulse_skip_cache_put(pulse_stage* st, int32_t mb, int32_t slot,
                                  const void* src, void* stream);

/* Copy the activation (stage dtype) or gradient (fp32) entry of (mb, slot)
 * into `dst` and mark it absent.  PULSE_E_CACHE_MISS if absent.  A
 * microbatch that never ran a forward is released once its last entry has
 * been taken. */
pulse_status pulse_skip_cache_take(pulse_stage* st, int32_t mb, int32_t slot,
                                   pulse_skip_kind kind, void* dst, void* stream);

/* *state = PULSE_SKIP_*_PRESENT bits of (mb, slot); 0 for an unknown mb. */
pulse_status pulse_skip_cache_state(const pulse_stage* st, int32_t mb, int32_t slot,
                                    int32_t* state);

/* Drop one microbatch / every in-flight microbatch (recovery primitive). */
pulse_status pulse_stage_release(pulse_stage* st, int32_t mb);
pulse_status pulse_stage_reset(pulse_stage* st);
int32_t pulse_stage_inflight(const pulse_stage* st);

/* Per-kernel timing: when enabled, every launch of the implicit-GEMM conv
 * kernel is bracketed by HIP events on the call's stream, and the backward
 * pass keeps all its work on that stream (no overlap with the
 * weight-gradient GEMMs, which otherwise run on an internal stream), so
 * the events time the kernel alone.  _read
 * synchronises those events and returns the launch count, the summed
 * duration in ms, the summed algorithmic FLOPs (2*M*N*K) and the summed
 * compulsory HBM bytes (each input element, weight and residual read once,
 * each output written once) since the last reset; any output pointer may
 * be NULL. */
pulse_status pulse_stage_timing(pulse_stage* st, int32_t enable);
pulse_status pulse_stage_timing_read(pulse_stage* st, int64_t* launches,
                                     double* ms, double* flops, double* bytes);

/* FLOPs of one microbatch's ENC+DEC forward and backward as 2*M*N*K summed
 * over every conv (forward, data gradient, weight gradient) and the
 * timestep linear. */
double pulse_stage_flops(const pulse_stage* st);

/* ---- pipeline schedule (Sec. V) ----------------------------------------
 *
 * A model cut into P = 2D partitions runs on D devices; partition p and its
 * skip partner P-1-p are collocated (Sec. IV-B) together with their
 * backward passes, so device q holds the skip-collocated stage made of
 * encoder partition q and decoder partition 2D-1-q (Sec. V-B; one
 * pulse_stage).  One microbatch is the chain of S = 4D unit-time stages
 * s = 0..P-1 (forward of partition s) and s = P..2P-1 (backward of partition
 * 2P-1-s).  A schedule is a table[d * T + t] over devices d and steps t
 * holding s * M + m (stage s of microbatch m) or -1 (idle); the caller owns
 * it.  Stage-to-device placement is the symmetric one: pair q on device q. */

/* Build the wave schedule of (D, M) (Sec. V-A objective: fewest steps).
 * Candidates are two list schedules (each step, every device runs one
 * runnable stage: backward-first deepest-first, or forward-first
 * deepest-first) and, for D <= 4 and a state space of at most 2e5 progress
 * vectors, an exact minimum found by breadth-first search over the
 * microbatches each stage has finished.  The fewest steps win, then the
 * fewest microbatches in flight on any device; *exact = 1 when the search
 * ran, so that the result is a proven minimum.  With table == NULL only *T
 * (the number of steps) is returned; otherwise table must hold D * cap
 * entries with cap >= *T (else PULSE_E_SHAPE) and receives the schedule as
 * table[d * T + t].  PULSE_E_INVALID_ARG for D outside [1, 64], M outside
 * [1, 4096] or T == NULL. */
pulse_status pulse_sched_build(int32_t D, int32_t M, int32_t* table, int32_t cap, int32_t* T,
                               int32_t* exact);

/* Check a schedule against the constraints of the scheduling formulation
 * (Sec. V-A): *violated receives a bit mask with bit k set when constraint
 * (k) fails -- (1) unique assignment, (3) fixed device mapping, (4)
 * collocation of the four stages of a skip pair, (5) sequential execution,
 * (6) monotonic microbatch order -- and bit 0 when the first stage is not on
 * device 0.  (2), one stage per device and step, holds by the table's
 * shape.  0 means valid. */
pulse_status pulse_sched_check(int32_t D, int32_t M, const int32_t* table, int32_t T,
                               int32_t* violated);

/* Microbatches each device holds at once under a schedule: peak[d] (D
 * entries, caller-owned) receives the largest number of microbatches whose
 * encoder forward on device d has run and whose encoder backward has not,
 * which is the max_inflight that device's stage needs. */
pulse_status pulse_sched_inflight(int32_t D, int32_t M, const int32_t* table, int32_t T,
                                  int32_t* peak);

/* Per-microbatch boundary tensors of one device (device pointers in the
 * stage dtype unless noted): x (encoder input), u (decoder upstream input),
 * temb, g_enc and g_dec (output gradients) in; y_enc, y_dec, dx, du out;
 * dtemb (fp32, accumulated) may be NULL. */
typedef struct {
  const void* x;
  const void* u;
  const void* temb;
  const void* g_enc;
  const void* g_dec;
  void* y_enc;
  void* y_dec;
  void* dx;
  void* du;
  float* dtemb;
} pulse_mb_io;

/* Execute steps [t0, t1) of device d's row of a schedule on its stage: each
 * cell becomes pulse_stage_forward/backward of the stage's ENC half (stage
 * s = d forward, s = 4D-1-d backward) or DEC half (s = 2D-1-d forward,
 * s = 2D+d backward) for that microbatch, in step order, on `stream` (io: M
 * entries, read only for the microbatches the steps touch).  A host runtime
 * that moves boundary tensors between devices calls it one step at a time
 * and exchanges at the step boundaries; one call over [0, T) runs the whole
 * row when all inputs are already resident.  The stage needs max_inflight
 * >= the microbatches the row keeps in flight.  PULSE_E_INVALID_ARG when
 * 0 <= t0 <= t1 <= T fails or a cell in the range is not one of the device's
 * four stages (nothing is enqueued then); otherwise the first failing stage
 * call's status. */
pulse_status pulse_sched_run_device(pulse_stage* st, int32_t D, int32_t d, int32_t M,
                                    const int32_t* table, int32_t T, int32_t t0, int32_t t1,
                                    const pulse_mb_io* io, void* stream);

/* Measurement helper, not part of the method: `blocks` workgroups of 256
 * threads each run `iters` iterations of independent bf16 MFMAs of the given
 * shape (32: 32x32x16, 16: 16x16x32) on register operands, with no memory
 * traffic in the loop.  `out` is caller-owned device memory of
 * blocks * 256 floats (one value per thread, kept so the chain is not
 * removed); *flops receives the FLOPs of the launch.  The caller times the
 * launch on `stream`.  PULSE_E_INVALID_ARG for a bad shape, count or NULL out;
 * PULSE_E_HIP if the launch fails. */
pulse_status pulse_mfma_probe(int32_t shape, int32_t blocks, int32_t iters, float* out,
                              double* flops, void* stream);

/* Thread-local description of the last error; valid until the next call. */
const char* pulse_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* PULSE_STAGE_H */
