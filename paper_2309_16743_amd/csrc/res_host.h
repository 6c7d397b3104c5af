// Host side of a reservoir's call sequence, free of HIP so that it can also be
// built for the CPU alone (the thread-sanitizer test drives it from many
// threads).  It holds the state that the calls' kernels take as arguments and
// that the order of the calls alone determines: the ticket counter, the number
// of stored samples N, the FIFO / FIRO ring positions and whether reception
// is over.  Every function runs under the reservoir's mutex.  *_admit decide
// from the state without changing it; *_commit take the call's ticket and
// advance the state, and are called only once the caller's earlier work is
// ordered before the call on the reservoir's stream, so that a call that
// fails before that point leaves the ticket sequence unchanged.
//
// Why N is host-known (Algorithm 1, Sec. 3.2.3): a Reservoir put of k rows
// leaves N = min(C, N + k), since every accepted row fills a free slot or
// replaces a seen sample and a = min(k, C - U) >= min(k, C - N); a FIFO /
// FIRO put accepts min(k, C - N); a batch that takes samples out (FIFO /
// FIRO, or any policy after reception ended) removes min(b, N).
#pragma once

#include <algorithm>
#include <cstdint>

#include "reservoir.h"

namespace ot {

struct ResSeq {
  int32_t policy = OT_POLICY_RESERVOIR;
  int64_t C = 0;
  int64_t T = 0;                 // threshold (0 once reception is over)
  uint64_t next_ticket = 0;
  int64_t n_host = 0;            // N
  int64_t occ_base = 0;          // ring position of the list's first entry (drain, FIFO, FIRO)
  int64_t free_head = 0;         // ring position of the first free slot (FIFO, FIRO)
  bool reception_over = false;
};

// What one put's kernels need from the host.
struct PutCall {
  uint64_t ticket = 0;
  int64_t n_before = 0;          // N before the call
  int64_t accepted = -1;         // FIFO / FIRO: min(k, C - N); Reservoir: decided on the device (-1)
  int may_evict = 0;             // Reservoir: N + k > C (the seen slots are indexed only then)
  int64_t free_head = 0;         // FIFO / FIRO: first free ring position before the call
};

inline int put_admit(const ResSeq& q) { return q.reception_over ? OT_E_CLOSED : OT_OK; }

inline PutCall put_commit(ResSeq& q, int64_t k) {
  PutCall c;
  c.ticket = q.next_ticket++;
  c.n_before = q.n_host;
  c.free_head = q.free_head;
  if (q.policy != OT_POLICY_RESERVOIR) {
    c.accepted = std::min<int64_t>(k, q.C - q.n_host);
    q.n_host += c.accepted;
    q.free_head = (q.free_head + c.accepted) % q.C;
  } else {
    c.may_evict = (q.n_host + k > q.C) ? 1 : 0;
    q.n_host = std::min<int64_t>(q.C, q.n_host + k);
  }
  return c;
}

// What one batch's kernels need from the host.
struct DrawCall {
  uint64_t ticket = 0;
  int64_t n_before = 0;          // N before the call
  int64_t drawn = 0;             // samples returned (b, or min(b, N) for a take)
  bool take = false;             // the drawn samples leave the buffer
  int64_t occ_base = 0;          // take: the list's first ring position before the call
  int64_t free_tail = 0;         // take: ring position after the free queue's last entry
};

// Whether a batch of b may be drawn now: OT_OK (with *drawn), OT_NOT_READY or
// OT_EMPTY.  Reservoir: N > T (Algorithm 1 waits while N <= T); FIFO: N >= b;
// FIRO: N > T and N >= b; after reception ended: N > 0, the batch is short
// when fewer than b remain.
inline int draw_admit(const ResSeq& q, int64_t b, int64_t* drawn) {
  *drawn = b;
  if (q.reception_over) {
    if (q.n_host == 0) return OT_EMPTY;
    *drawn = std::min<int64_t>(b, q.n_host);
    return OT_OK;
  }
  if (q.policy == OT_POLICY_FIFO) return q.n_host < b ? OT_NOT_READY : OT_OK;
  if (q.policy == OT_POLICY_FIRO) return (q.n_host <= q.T || q.n_host < b) ? OT_NOT_READY : OT_OK;
  return q.n_host <= q.T ? OT_NOT_READY : OT_OK;
}

inline DrawCall draw_commit(ResSeq& q, int64_t drawn) {
  DrawCall c;
  c.ticket = q.next_ticket++;
  c.n_before = q.n_host;
  c.drawn = drawn;
  c.take = q.reception_over || q.policy != OT_POLICY_RESERVOIR;
  if (c.take) {
    c.occ_base = q.occ_base;
    c.free_tail = (q.free_head + q.C - q.n_host) % q.C;   // C - N entries follow the free queue's head
    q.occ_base = (q.occ_base + drawn) % q.C;
    q.n_host -= drawn;
  }
  return c;
}

// End of reception (the drain of Sec. 3.2.3): the threshold drops to 0; a
// Reservoir's list of stored samples restarts at ring position 0 (slots
// [0, N) in order).  Returns OT_E_STATE when reception is already over.
inline int end_commit(ResSeq& q) {
  if (q.reception_over) return OT_E_STATE;
  q.reception_over = true;
  q.T = 0;
  if (q.policy == OT_POLICY_RESERVOIR) q.occ_base = 0;
  return OT_OK;
}

}  // namespace ot
