/* GPU-resident training buffer (Sec. 3.2.3), one per device: the paper's
 * Algorithm 1 "Reservoir" (the default policy), or one of its two comparison
 * buffers, FIFO and FIRO, which evict a sample when it is read (see
 * ot_reservoir_policy below).
 *
 * The buffer holds at most C samples, each an input row x (x_dim fp32: the
 * simulation parameters X and the time t, Sec. 4.1) and a field row u (u_dim
 * fp32: the discretised u_X^t).  A sample is "unseen" until it is first drawn
 * into a batch and "seen" afterwards.  put() stores new samples, replacing
 * uniformly chosen seen samples once the buffer is full and never discarding
 * unseen ones; sample_batch() draws B slots uniformly with replacement over all
 * stored samples, but only while more than T samples are stored; after
 * reservoir_end_reception() the threshold is lifted and every draw removes its
 * sample until the buffer is empty.
 *
 * Randomness: every draw is output word 0 of Philox4x64-10 (Salmon et al.,
 * SC'11) with key (seed, 0) and counter (j, ticket, kind, 0), mapped onto
 * [0, n) as floor(w * n / 2^64); kind 1 = batch draw, 2 = eviction draw.
 * Tickets number the state-changing calls of one reservoir 0, 1, 2, ... in the
 * order the calls acquire the reservoir's lock; refused calls, and calls that
 * fail before enqueueing any work, take no ticket.
 * Results depend only on (seed, the sequence of calls in ticket order).
 *
 * Memory and streams: the reservoir owns its device memory (slabs, per-slot
 * seen counts and sample ids, counters).  All work runs on one ordering
 * stream, in ticket order.  Every call takes the caller's stream: the
 * ordering stream first waits for work already queued on the caller's stream,
 * and the caller's stream then waits for the call's work, so buffers passed
 * in may be reused in stream order.  When the caller's stream is the ordering
 * stream no events are used.  Calls are asynchronous unless stated.  Reservoir
 * calls are thread-safe.
 *
 * Device pointers must be 16-byte aligned and their leading dimensions (in
 * elements) multiples of 4 where a field row is involved.
 */
#ifndef OT_RESERVOIR_H
#define OT_RESERVOIR_H

#include <stdint.h>

#include "ot_status.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ot_reservoir ot_reservoir;

/* Counters of one reservoir, read after all its queued work completed. */
typedef struct ot_reservoir_stats {
  int64_t capacity;       /* C */
  int64_t threshold;      /* T (0 after end_reception) */
  int64_t n;              /* stored samples N = unseen + seen */
  int64_t unseen;         /* U */
  int64_t seen;           /* S */
  int64_t total_put;      /* accepted samples */
  int64_t total_evicted;  /* seen samples replaced by puts */
  int64_t total_deleted;  /* samples removed by draws after end_reception */
  int64_t total_draws;    /* samples handed out in batches */
  int64_t next_ticket;
  int64_t next_sample_id;
  int32_t reception_over;
  int32_t hist_len;       /* length of the eviction histogram (reservoir_read_meta) */
  int32_t policy;         /* ot_reservoir_policy */
  int32_t reserved;
} ot_reservoir_stats;

/* Buffer policies (Sec. 3.2.3).  Each answers put / sample_batch /
 * end_reception over the same slabs, tickets, statuses and gather.
 * OT_POLICY_RESERVOIR: Algorithm 1 as described below (evict seen samples on
 *   write, draw with replacement while N > T, drain after reception).
 * OT_POLICY_FIFO: first in, first out.  put accepts a = min(k, C - N) (the
 *   paper suspends production while the buffer is full); a batch takes the b
 *   oldest samples and removes them, and is refused (OT_NOT_READY) while
 *   N < b -- a batch as soon as the buffer holds one; the threshold is not
 *   used.  Every sample is used exactly once, in arrival order.
 * OT_POLICY_FIRO: first in, random out.  put as FIFO (appends to the list of
 *   stored samples); a batch is refused while N <= T or N < b, otherwise it
 *   takes b distinct samples by partial Fisher-Yates over the list (Philox
 *   kind 1, j = draw index, range N - j; the remaining list keeps the
 *   shuffled order) and removes them.
 * FIFO and FIRO: after end_reception the threshold is 0, the last batch may be
 *   short (min(b, N)) and an empty buffer answers OT_EMPTY; b <= 4096; a freed
 *   slot joins a queue of free slots and a stored row takes the queue's head
 *   (initially slots 0 .. C-1 in order, so FIFO fills the slab as a ring);
 *   nothing is evicted by a put, so total_evicted stays 0 and every sample
 *   leaves with seen count 1. */
enum ot_reservoir_policy { OT_POLICY_RESERVOIR = 0, OT_POLICY_FIFO = 1, OT_POLICY_FIRO = 2 };

/* Create a reservoir of `capacity` samples of x_dim + u_dim fp32 values.
 * threshold: batches are refused while N <= threshold (Algorithm 1, get;
 * unused by FIFO).  seed: Philox key word 0.  policy: ot_reservoir_policy.
 * order_stream: hipStream_t to run the reservoir's
 * work on, or NULL to let the reservoir create (and later destroy) its own.
 * Allocates C * (round_up(x_dim, 4) + round_up(u_dim, 64)) * 4 bytes of slab
 * plus 20 bytes per slot of metadata on the current device.
 * Errors: OT_E_INVAL (capacity < 1 or > 2^31-1, threshold < 0, x_dim or u_dim
 * < 1, unknown policy), OT_E_NOMEM, OT_E_HIP. */
int reservoir_create(ot_reservoir** out, int64_t capacity, int64_t threshold,
                     int64_t x_dim, int64_t u_dim, uint64_t seed, int32_t policy,
                     void* order_stream);

/* Store up to k samples (Algorithm 1, put; Sec. 3.2.3).
 * x: k rows of x_dim fp32 at stride ldx elements (may be NULL: x rows are
 * then stored as zeros); u: k rows of u_dim fp32 at stride ldu elements (ldu
 * a multiple of 4, u 16-byte aligned).  Accepts the in-order prefix
 * a = min(k, C - U) (the paper's put blocks while unseen samples fill the
 * buffer; here the caller re-offers the rest later).  Rows go to free slots
 * first (ascending), then replace seen samples picked by a partial
 * Fisher-Yates shuffle over the ascending list of seen slots (Philox kind 2,
 * j = replacement index); row F + j replaces victim j.  Each stored row gets
 * the next sample id and a seen count of 0.
 * accepted_dev: device int64 that receives a when the work runs (nullable).
 * A buffer full of unseen samples (U = C) accepts a = 0: that "full" answer
 * arrives only through accepted_dev; the status is still OT_OK, because U
 * changes on the device and the host does not know it when the call returns.
 * ticket_out: host uint64 that receives the call's ticket (nullable).
 * FIFO / FIRO accept a = min(k, C - N) into the free slots (see above).
 * k may be 0 (takes a ticket, stores nothing).  1 <= k <= 4096 otherwise.
 * Errors: OT_E_CLOSED after end_reception, OT_E_INVAL, OT_E_HIP. */
int reservoir_put(ot_reservoir* r, const float* x, int64_t ldx, const float* u, int64_t ldu,
                  int64_t k, void* stream, int64_t* accepted_dev, uint64_t* ticket_out);

/* Draw a batch of b samples (Algorithm 1, get, repeated b times).
 * Normal phase: returns OT_NOT_READY (no ticket, nothing enqueued) while
 * N <= T; otherwise draw j picks slot floor(w_j * N / 2^64) with
 * w_j = Philox(seed; j, ticket, 1), with replacement; a slot drawn for the
 * first time becomes seen; every draw adds one to the slot's seen count.
 * After end_reception: returns OT_EMPTY when N == 0; otherwise draws
 * b' = min(b, N) distinct samples by partial Fisher-Yates over the stored
 * samples and removes them (the last batch may be short; *count_out = b').
 * slots: device int32[b], receives the drawn slots (required).
 * x_out: device fp32 b rows at stride ldxo (nullable: not gathered).
 * u_out: device fp32 b rows at stride lduo (nullable; lduo multiple of 4).
 * count_out: host int64 receiving the number of rows drawn (nullable).
 * The batch is atomic with respect to puts.
 * FIFO / FIRO: see ot_reservoir_policy.
 * Errors: OT_E_INVAL (b < 1, b > 65536 (4096 for FIFO / FIRO and while
 * draining), null slots, bad ld), OT_E_HIP. */
int reservoir_sample_batch(ot_reservoir* r, int64_t b, void* stream, int32_t* slots,
                           float* x_out, int64_t ldxo, float* u_out, int64_t lduo,
                           int64_t* count_out, uint64_t* ticket_out);

/* Mark reception as over (the paper's is_reception_over): later puts fail
 * with OT_E_CLOSED, the threshold becomes 0 and later batches drain the
 * buffer.  Takes no ticket (it draws nothing).  Errors: OT_E_STATE if
 * already over. */
int reservoir_end_reception(ot_reservoir* r);

/* Device addresses of the slabs, for callers that read stored rows in place
 * (a train step whose targets are the u rows of the drawn slots): the row of
 * slot k is x + k * ldx (x_dim fp32) and u + k * ldu (u_dim fp32); the
 * addresses stay valid until reservoir_destroy.  A slot's rows change only
 * when a put stores a sample into it, so a caller that reads rows must order
 * the puts that follow its reads after them (for instance by passing puts a
 * stream that has waited for an event recorded after the reads).  Each
 * pointer argument is nullable.  Errors: OT_E_INVAL (NULL reservoir). */
int reservoir_slab(ot_reservoir* r, const float** x, int64_t* ldx, const float** u, int64_t* ldu);

/* Synchronise with the reservoir's queued work and read its counters. */
int reservoir_stats(ot_reservoir* r, ot_reservoir_stats* out);

/* Synchronise and copy per-slot metadata to host memory (each pointer
 * nullable): seen_count int32[C] (-1 for an empty slot), sample_id int64[C]
 * (-1 for an empty slot), evict_hist int64[hist_len]: number of samples that
 * left the buffer (evicted or drained) with seen count k, the last bucket
 * counting all k >= hist_len - 1. */
int reservoir_read_meta(ot_reservoir* r, int32_t* seen_count, int64_t* sample_id,
                        int64_t* evict_hist);

/* Synchronise and copy stored rows of the given slots to host memory
 * (test and checkpoint hook).  x_host: n x x_dim, u_host: n x u_dim, dense. */
int reservoir_read_rows(ot_reservoir* r, const int32_t* slots_host, int64_t n,
                        float* x_host, float* u_host);

/* Checkpoint / restore (the paper's server is checkpointed regularly and a
 * failed server restarts from its last checkpoint, Sec. 3.1).  Synchronous:
 * both wait for the reservoir's queued work.  The checkpoint is a host blob
 * holding the policy, shape, threshold, seed, ticket counter, counters,
 * eviction histogram, per-slot metadata, list and free-slot rings, and the
 * x and u rows of every stored sample; restoring it into a reservoir created
 * with the same capacity, x_dim, u_dim and policy reproduces the state, so
 * later calls with the same tickets give the same slots and rows as the
 * reservoir that was checkpointed.
 * reservoir_checkpoint_size: *bytes = blob size for the current state.
 * reservoir_checkpoint: writes the blob into buf (caller-owned host memory
 *   of at least that size).  Errors: OT_E_INVAL (buffer too small), OT_E_HIP.
 * reservoir_restore: replaces the reservoir's state with the blob's.
 *   Errors: OT_E_INVAL (not a reservoir checkpoint, other shape or policy,
 *   truncated or inconsistent blob: nothing is changed), OT_E_HIP. */
int reservoir_checkpoint_size(ot_reservoir* r, int64_t* bytes);
int reservoir_checkpoint(ot_reservoir* r, void* buf, int64_t bytes);
int reservoir_restore(ot_reservoir* r, const void* buf, int64_t bytes);

/* Kernel phases of the reservoir calls, for the timing hook below. */
enum ot_reservoir_phase {
  OT_PH_PUT_ASSIGN = 0,  /* put: slot assignment and eviction draws */
  OT_PH_PUT_COPY = 1,    /* put: row copies into the slabs */
  OT_PH_SELECT = 2,      /* sample: batch draws and seen-count update */
  OT_PH_GATHER = 3,      /* sample: row copies into the batch buffers */
  OT_RESERVOIR_PHASES = 4
};

/* Profiling hook: time the kernels of every phase in phase_mask for the next
 * max_calls put or sample calls with HIP events on the ordering stream.  The
 * single-kernel phases PUT_COPY and GATHER hand their events to the launch
 * (hipExtLaunchKernel), which stamps them with the kernel's own start and
 * end; the others record events before and after their kernels.  Allocates 2
 * events per phase and call. */
int reservoir_timing_begin(ot_reservoir* r, uint32_t phase_mask, int64_t max_calls);

/* Wait for the recorded events and return summed milliseconds and counts per
 * phase (arrays of OT_RESERVOIR_PHASES, each nullable). */
int reservoir_timing_end(ot_reservoir* r, double* ms_total, int64_t* count);

/* Synchronise and free everything the reservoir owns. */
int reservoir_destroy(ot_reservoir* r);

#ifdef __cplusplus
}
#endif

#endif /* OT_RESERVOIR_H */
