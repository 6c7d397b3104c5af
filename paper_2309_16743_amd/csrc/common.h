// Internal helpers of the online-training library: error state, HIP checks,
// small device utilities.  Not part of the public C ABI.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <cstdarg>
#include <string>
#include <vector>

#include "ot_status.h"

namespace ot {

// Record a message for ot_last_error() on this thread and return `code`.
int set_error(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();

inline int64_t round_up(int64_t v, int64_t m) { return (v + m - 1) / m * m; }

// Per-phase HIP-event timing of the kernels one call enqueues (profiling
// hook).  begin() creates start/end events for max_calls calls of every phase
// in `mask`; mark() records them on the stream the phase's kernels use;
// end() waits for the events and returns the summed milliseconds per phase.
struct PhaseTimer {
  uint32_t mask = 0;
  int nph = 0;
  int64_t max_calls = 0;
  int64_t call = 0;
  std::vector<hipEvent_t> ev;
  std::vector<char> rec;

  bool on(int phase) const { return mask && ((mask >> phase) & 1u) && call < max_calls; }
  void mark(hipStream_t st, int phase, int which) {
    if (!on(phase)) return;
    const size_t i = (size_t)((call * nph + phase) * 2 + which);
    if (hipEventRecord(ev[i], st) == hipSuccess) rec[i] = 1;
  }
  // Start and stop events of a phase that is a single kernel, for
  // hipExtLaunchKernelGGL: the runtime then stamps them with that kernel's own
  // start and end (mark() around a launch also counts the dispatch gap before
  // the kernel).  Both stay null while the phase is not timed.
  void kernel_events(int phase, hipEvent_t* start, hipEvent_t* stop) {
    *start = *stop = nullptr;
    if (!on(phase)) return;
    const size_t i = (size_t)((call * nph + phase) * 2);
    *start = ev[i];
    *stop = ev[i + 1];
    rec[i] = rec[i + 1] = 1;
  }
  void next_call() {
    if (mask) ++call;
  }
  int begin(uint32_t m, int phases, int64_t calls);
  int end(double* ms, int64_t* counts);
  void release();
};
inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Sequential writer / reader of a checkpoint blob in caller-owned host memory.
// Every access is bounds-checked; ok() turns false at the first overrun and
// later accesses do nothing.
struct BlobWriter {
  unsigned char* p;
  int64_t cap, off = 0;
  bool good = true;
  BlobWriter(void* buf, int64_t bytes) : p(static_cast<unsigned char*>(buf)), cap(bytes) {}
  unsigned char* take(int64_t n) {
    if (!good || n < 0 || off + n > cap) { good = false; return nullptr; }
    unsigned char* q = p + off;
    off += n;
    return q;
  }
  template <class T> void put(const T& v) {
    if (unsigned char* q = take(sizeof(T))) __builtin_memcpy(q, &v, sizeof(T));
  }
};
struct BlobReader {
  const unsigned char* p;
  int64_t cap, off = 0;
  bool good = true;
  BlobReader(const void* buf, int64_t bytes) : p(static_cast<const unsigned char*>(buf)), cap(bytes) {}
  const unsigned char* take(int64_t n) {
    if (!good || n < 0 || off + n > cap) { good = false; return nullptr; }
    const unsigned char* q = p + off;
    off += n;
    return q;
  }
  template <class T> T get() {
    T v{};
    if (const unsigned char* q = take(sizeof(T))) __builtin_memcpy(&v, q, sizeof(T));
    return v;
  }
};

}  // namespace ot

// Evaluate a HIP call; on failure record the message and return OT_E_HIP.
#define OT_HIP(call)                                                                    \
  do {                                                                                  \
    hipError_t e_ = (call);                                                             \
    if (e_ != hipSuccess)                                                               \
      return ot::set_error(OT_E_HIP, "%s failed: %s", #call, hipGetErrorString(e_));    \
  } while (0)

// Check the last kernel launch.
#define OT_LAUNCHED(name)                                                               \
  do {                                                                                  \
    hipError_t e_ = hipGetLastError();                                                  \
    if (e_ != hipSuccess)                                                               \
      return ot::set_error(OT_E_HIP, "launch of %s failed: %s", name,                   \
                           hipGetErrorString(e_));                                      \
  } while (0)

#define OT_REQUIRE(cond, ...)                                                           \
  do {                                                                                  \
    if (!(cond)) return ot::set_error(OT_E_INVAL, __VA_ARGS__);                         \
  } while (0)

// Device helpers -------------------------------------------------------------------
namespace ot {
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
}  // namespace ot

#ifdef __HIPCC__
namespace ot {

__device__ inline float warp_sum(float v) {
  // Fixed butterfly order over the 64 lanes of a wavefront: deterministic.
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

__device__ inline double warp_sum(double v) {
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

}  // namespace ot
#endif
