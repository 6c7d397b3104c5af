/* Fully-connected deep surrogate and its train step (the paper's use case,
 * Sec. 4.1): an MLP that maps the 6 inputs (X, t) to the whole field u_X^t
 * (Eq. 1 defines the mapping X -> {u_X^t}), ReLU on hidden layers, identity
 * output, mean-squared-error loss, Adam with learning rate 1e-3.
 *
 * Layer l (1..L) has W_l of widths[l] x widths[l-1] (out x in, row-major)
 * and b_l of widths[l]; Z_l = A_{l-1} W_l^T + b_l, A_l = ReLU(Z_l) for l < L,
 * Y = Z_L.  Loss = mean over the B x D batch of (Y - U)^2.  Adam (Kingma and
 * Ba, 2015): beta1, beta2, eps as given, bias-corrected, no weight decay, step
 * counter t from 1, in the operation order
 *   m = b1 m + (1 - b1) g;  v = b2 v + (1 - b2) g^2;
 *   p = p - lr (m / (1 - b1^t)) / (sqrt(v / (1 - b2^t)) + eps).
 * ReLU'(0) = 0.
 *
 * Precision OT_FP32: every GEMM on fp32 operands with fp32 accumulation.
 * Precision OT_BF16: layer 1 (K = widths[0]) in fp32; every other GEMM takes
 * bf16 operands (activations, a bf16 copy of W refreshed by each Adam step,
 * and back-propagated dY / dZ), accumulates in fp32; master weights, Adam
 * moments and gradients stay fp32.
 *
 * Initialisation: W and b ~ U(-1/sqrt(fan_in), 1/sqrt(fan_in)); element e of
 * layer l (flat index over W then b) is (2 m / 2^24 - 1) / sqrt(fan_in) rounded
 * to fp32, m = top 24 bits of Philox4x64-10 word 0 at counter (e, l-1, 3, 0),
 * key (seed, 0).
 *
 * Ownership: the surrogate owns its parameters, gradients, Adam state and
 * workspaces (device memory on the device current at creation).  Device
 * pointers passed in are the caller's; they must be 16-byte aligned and field
 * rows must have leading dimensions that are multiples of 4.  Calls on one
 * surrogate must not overlap (one training thread, as in the paper's server);
 * train_step and predict are asynchronous on the given stream.
 */
#ifndef OT_SURROGATE_H
#define OT_SURROGATE_H

#include <stdint.h>

#include "ot_status.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ot_surrogate ot_surrogate;

enum ot_precision { OT_FP32 = 0, OT_BF16 = 1 };

/* Creation flags.
 * OT_SURROGATE_KEEP_GRADS: store every gradient of a train step, then run
 *   Adam over all parameters in one pass.  Without it (the default) the
 *   output layer's weights are updated by Adam inside the epilogue of their
 *   weight-gradient GEMM (or of its split-K reduction), which runs after the
 *   output layer's input gradient has read the old weights: that gradient
 *   (widths[L] x widths[L-1] fp32, the largest array of the step) is never
 *   written or read back, and surrogate_get_grads refuses it.  Both modes
 *   apply the same Adam arithmetic to the same gradient sums. */
enum ot_surrogate_flags { OT_SURROGATE_KEEP_GRADS = 1 };

/* Create an MLP with n_widths - 1 layers (2 <= n_widths <= 16, every width in
 * [1, 2^26]), parameters initialised from `seed` as above, Adam state zero.
 * max_batch: rows the train / predict workspaces are first sized for (grown
 * on demand).  flags: 0 or OT_SURROGATE_KEEP_GRADS.
 * Errors: OT_E_INVAL, OT_E_NOMEM, OT_E_HIP. */
int surrogate_create(ot_surrogate** out, const int64_t* widths, int32_t n_widths,
                     int32_t precision, float lr, float beta1, float beta2, float eps,
                     uint64_t seed, int64_t max_batch, uint32_t flags);

/* Replace layer `layer` (0-based) parameters from dense host arrays W
 * (widths[layer+1] x widths[layer]) and b (widths[layer+1]); either may be
 * NULL.  Synchronous.  Refreshes the bf16 weight copy. */
int surrogate_set_params(ot_surrogate* s, int32_t layer, const float* W_host, const float* b_host);

/* Copy layer parameters (fp32 master) to dense host arrays.  Synchronous. */
int surrogate_get_params(ot_surrogate* s, int32_t layer, float* W_host, float* b_host);

/* Copy the gradients of the last train step of one layer.  Synchronous.
 * OT_E_STATE for the output layer's dW_host (non-NULL) when that step fused
 * the output layer's Adam update (no OT_SURROGATE_KEEP_GRADS). */
int surrogate_get_grads(ot_surrogate* s, int32_t layer, float* dW_host, float* db_host);

/* Copy Adam moments of one layer and the step counter t (each nullable). */
int surrogate_get_adam_state(ot_surrogate* s, int32_t layer, float* mW_host, float* mb_host,
                             float* vW_host, float* vb_host, int64_t* t_out);

/* Set the learning rate used by later train steps (schedules). */
int surrogate_set_lr(ot_surrogate* s, float lr);

/* Device step counter, for callers that capture a train step once (HIP graph
 * capture on their stream) and replay it.  Adam's bias corrections
 * 1 - beta^t (Kingma and Ba's Algorithm 1, the optimizer of Sec. 4.1) depend
 * on the step t, normally a host-side argument of the step's kernels; with
 * enable = 1 the kernels read the number of completed steps from device
 * memory instead and the step ends with a launch that advances it, so that
 * the captured launches stay valid for every replay.  The corrections are
 * formed the same way in both modes (binary exponentiation in double), so
 * steps agree bit for bit.  Switching synchronises the device; with the
 * counter on, surrogate_get_adam_state and surrogate_checkpoint read the
 * device's count, surrogate_restore sets it, and enable = 0 copies it back to
 * the host.  A captured step also fixes the learning rate, the batch size,
 * the buffers and the stream it was captured with.  Errors: OT_E_INVAL,
 * OT_E_NOMEM, OT_E_HIP. */
int surrogate_set_device_step(ot_surrogate* s, int32_t enable);

/* One train step on a batch of b rows: forward, MSE loss, backward, Adam.
 * x: b rows of widths[0] fp32 at stride ldx; u: b target rows of widths[L]
 * fp32 at stride ldu (multiple of 4).  loss_dev: device fp32 scalar that
 * receives the batch loss (nullable).  1 <= b <= 2^20.
 * Errors: OT_E_INVAL, OT_E_NOMEM, OT_E_HIP. */
int surrogate_train_step(ot_surrogate* s, const float* x, int64_t ldx, const float* u,
                         int64_t ldu, int64_t b, void* stream, float* loss_dev);

/* The same train step with the targets read in place from a larger array
 * (the reservoir's u slab, reservoir_slab), so that a batch needs no copy of
 * its field rows: target row j is u + rows[j] * ldu.  rows: device int32[b]
 * (4-byte aligned), each in [0, n_rows); an index outside that range is
 * clamped into it on the device (a wrong row is read, never memory outside
 * the array).  x, ldx, b, stream, loss_dev as for surrogate_train_step.
 * targets_read: hipEvent_t recorded on `stream` as soon as every target row
 * has been read (after the output layer's forward), so that a producer may
 * overwrite the rows after it while the rest of the step runs; nullable.
 * Results are those of surrogate_train_step on the gathered rows, bit for bit.
 * Errors: OT_E_INVAL (as surrogate_train_step; NULL or misaligned rows,
 * n_rows < 1), OT_E_NOMEM, OT_E_HIP. */
int surrogate_train_step_rows(ot_surrogate* s, const float* x, int64_t ldx, const float* u,
                              int64_t ldu, const int32_t* rows, int64_t n_rows, int64_t b, void* stream,
                              float* loss_dev, void* targets_read);

/* Surrogate prediction Y = f_theta(x) (Eq. 1's u_X^t estimate) for n rows.
 * x: n rows at stride ldx; y: n rows of widths[L] fp32 at stride ldy
 * (multiple of 4).  Errors: OT_E_INVAL, OT_E_NOMEM, OT_E_HIP. */
int surrogate_predict(ot_surrogate* s, const float* x, int64_t ldx, int64_t n, float* y,
                      int64_t ldy, void* stream);

/* Prediction that allocates nothing, for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc.  Same arguments, checks and results as surrogate_predict
 * (bit for bit when n <= max_batch), but all n rows go through one forward
 * pass whose hidden activations and split-K partial products live in a
 * library-owned scratch array of OT_PREDICT_NOALLOC_SCRATCH_BYTES per device
 * (a static device array, held until the process ends) instead of the
 * surrogate's workspaces; the call never calls hipMalloc, hipFree or a
 * synchronising runtime function.  The scratch needs no clearing (every byte
 * a call reads, the same call wrote first).  Every call on one device shares
 * that device's scratch: calls that may overlap on one device (other streams,
 * other surrogates, other threads) race and must be ordered by the caller.
 * The surrogate's device must be current.  1 <= n <= 2^20 (n = 0 does
 * nothing); n must also fit the scratch: roughly n * (sum of the hidden
 * widths) * (4 bytes fp32, 2 bytes bf16) plus any split-K partials.
 * Errors: OT_E_INVAL (as surrogate_predict; n too large for the scratch, with
 * the bytes needed in the message), OT_E_STATE (another device is current),
 * OT_E_HIP. */
enum { OT_PREDICT_NOALLOC_SCRATCH_BYTES = 64 << 20 };
int surrogate_predict_noalloc(ot_surrogate* s, const float* x, int64_t ldx, int64_t n, float* y,
                              int64_t ldy, void* stream);

/* Validation loss (Sec. 4.4 validates on simulations never used for
 * training): the mean over n x widths[L] of (f_theta(x) - u)^2 with the
 * current parameters, by the train step's forward and fused-MSE kernels;
 * parameters, gradients and Adam state are untouched.  Rows are processed in
 * chunks of the workspace size and their squared residuals summed in fp64 in
 * a fixed order.  x: n rows at stride ldx; u: n target rows at stride ldu
 * (multiple of 4, 16-byte aligned); loss_dev: device fp32 scalar (required).
 * Asynchronous on `stream`; calls on one surrogate must not overlap.
 * Errors: OT_E_INVAL, OT_E_HIP. */
int surrogate_eval_loss(ot_surrogate* s, const float* x, int64_t ldx, const float* u,
                        int64_t ldu, int64_t n, void* stream, float* loss_dev);

/* Checkpoint / restore of the training state (Sec. 3.1: the server is
 * checkpointed and restarts from its last checkpoint).  Synchronous.  The
 * blob holds precision, widths, the Adam step counter and hyper-parameters,
 * and the fp32 parameters and both Adam moments; gradients are recomputed by
 * every step and the bf16 weight copy is rounded again from the master
 * weights, so a restored surrogate continues bit for bit.
 * surrogate_checkpoint_size: *bytes = blob size.
 * surrogate_checkpoint: writes the blob into buf (host, >= that size).
 * surrogate_restore: into a surrogate created with the same widths and
 *   precision.  Errors: OT_E_INVAL (buffer too small, not a surrogate
 *   checkpoint, other shape or precision: nothing is changed), OT_E_HIP. */
int surrogate_checkpoint_size(ot_surrogate* s, int64_t* bytes);
int surrogate_checkpoint(ot_surrogate* s, void* buf, int64_t bytes);
int surrogate_restore(ot_surrogate* s, const void* buf, int64_t bytes);

/* Kernel phases of one train step, for the timing hook below. */
enum ot_surrogate_phase {
  OT_PH_FWD_HIDDEN = 0,    /* hidden-layer forward GEMMs (bias + ReLU epilogue) */
  OT_PH_FWD_OUTPUT = 1,    /* output-layer forward GEMM with the fused MSE epilogue */
  OT_PH_LOSS = 2,          /* not recorded: the loss is reduced in the step's last pass */
  OT_PH_WGRAD_OUTPUT = 3,  /* output-layer weight-gradient GEMM (with bias gradient) */
  OT_PH_IGRAD_OUTPUT = 4,  /* output-layer input-gradient GEMM */
  OT_PH_IGRAD_REDUCE = 5,  /* split-K reduction + ReLU mask of that gradient */
  OT_PH_BWD_HIDDEN = 6,    /* hidden-layer backward */
  OT_PH_ADAM = 7,          /* the step's last pass (Adam over the parameters not updated in a fused
                              epilogue, and the loss); not recorded when that pass runs inside the
                              output layer's split-K Adam reduction (fp32, fused) */
  OT_PH_WGRAD_REDUCE = 8,  /* split-K reduction of the output-layer weight gradient (fused: with
                              Adam on W_L and b_L and the step's last pass) */
  OT_SURROGATE_PHASES = 9
};

/* Profiling hook: time every phase in phase_mask (bit p = phase p) for the
 * next max_steps train steps with HIP events on the stream each step runs on.
 * A phase that is one kernel launch (the output-layer GEMMs) passes its
 * events to that launch (hipExtLaunchKernel), so they take the kernel's own
 * start and end; other phases record events before and after their kernels,
 * which also counts the dispatch gaps.  Allocates 2 events per phase and
 * step. */
int surrogate_timing_begin(ot_surrogate* s, uint32_t phase_mask, int64_t max_steps);

/* Wait for the recorded events; ms_total[p] receives the summed duration of
 * phase p in milliseconds and count[p] the number of steps it covers
 * (arrays of OT_SURROGATE_PHASES, each nullable).  Releases the events. */
int surrogate_timing_end(ot_surrogate* s, double* ms_total, int64_t* count);

/* Synchronise and free everything the surrogate owns. */
int surrogate_destroy(ot_surrogate* s);

#ifdef __cplusplus
}
#endif

#endif /* OT_SURROGATE_H */
