/* Status codes and error reporting shared by every entry point of the
 * online-training library (training reservoir + surrogate train step).
 *
 * Every entry point is extern "C", never throws, and returns one of the codes
 * below.  A negative code is an error: the call enqueued nothing and left the
 * object unchanged (arguments are validated before any work is issued), except
 * OT_E_HIP, which reports a HIP runtime failure and may leave work partly
 * enqueued.  A positive code is a non-error refusal that mirrors one of the
 * waits of the paper's buffer (Algorithm 1 "Reservoir": a get waits while the
 * population is at or below the threshold; after reception ends the buffer
 * drains until empty).
 */
#ifndef OT_STATUS_H
#define OT_STATUS_H

#ifdef __cplusplus
extern "C" {
#endif

enum ot_status {
  OT_OK = 0,
  OT_NOT_READY = 1,  /* sample refused: population N <= threshold T */
  OT_EMPTY = 3,      /* sample refused: reception is over and N == 0 */
  OT_E_INVAL = -1,   /* bad argument (null handle, size, alignment, leading dimension) */
  OT_E_NOMEM = -2,   /* device allocation failed */
  OT_E_HIP = -3,     /* HIP runtime error; message in ot_last_error() */
  OT_E_CLOSED = -4,  /* put after reservoir_end_reception */
  OT_E_STATE = -5    /* call not valid in the object's current state */
};

/* Message describing the last non-OK status returned on the calling thread.
 * The string is owned by the library and valid until the next call on the
 * same thread.  Returns "" if the last call succeeded. */
const char* ot_last_error(void);

/* Library version string, e.g. "0.1.0 gfx950". Static storage. */
const char* ot_version(void);

#ifdef __cplusplus
}
#endif

#endif /* OT_STATUS_H */
