// Error state and version of the online-training library.
#include "common.h"

#include <cstdio>

namespace ot {

static thread_local std::string t_error;

int set_error(int code, const char* fmt, ...) {
  char buf[1024];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  t_error = buf;
  return code;
}

void clear_error() { t_error.clear(); }

void PhaseTimer::release() {
  for (hipEvent_t e : ev)
    if (e) (void)hipEventDestroy(e);
  ev.clear();
  rec.clear();
  mask = 0;
  call = 0;
  max_calls = 0;
}

int PhaseTimer::begin(uint32_t m, int phases, int64_t calls) {
  release();
  if (calls < 1 || calls > 100000) return set_error(OT_E_INVAL, "timing: max_calls outside [1, 100000]");
  nph = phases;
  ev.assign((size_t)(calls * phases * 2), nullptr);
  rec.assign(ev.size(), 0);
  for (int64_t c = 0; c < calls; ++c)
    for (int p = 0; p < phases; ++p)
      if ((m >> p) & 1u)
        for (int w = 0; w < 2; ++w) {
          hipError_t e = hipEventCreate(&ev[(size_t)((c * phases + p) * 2 + w)]);
          if (e != hipSuccess) {
            release();
            return set_error(OT_E_HIP, "hipEventCreate failed: %s", hipGetErrorString(e));
          }
        }
  mask = m;
  max_calls = calls;
  call = 0;
  return OT_OK;
}

int PhaseTimer::end(double* ms, int64_t* counts) {
  for (int p = 0; p < nph; ++p) {
    if (ms) ms[p] = 0.0;
    if (counts) counts[p] = 0;
  }
  const int64_t done = call < max_calls ? call : max_calls;
  for (int64_t c = 0; c < done; ++c)
    for (int p = 0; p < nph; ++p) {
      if (!((mask >> p) & 1u)) continue;
      const size_t ia = (size_t)((c * nph + p) * 2);
      if (!rec[ia] || !rec[ia + 1]) continue;
      hipEvent_t a = ev[ia], b = ev[ia + 1];
      hipError_t e = hipEventSynchronize(b);
      float t = 0.f;
      if (e == hipSuccess) e = hipEventElapsedTime(&t, a, b);
      if (e != hipSuccess) {
        release();
        return set_error(OT_E_HIP, "timing event failed: %s", hipGetErrorString(e));
      }
      if (ms) ms[p] += t;
      if (counts) counts[p] += 1;
    }
  release();
  return OT_OK;
}

}  // namespace ot

extern "C" const char* ot_last_error(void) { return ot::t_error.c_str(); }

extern "C" const char* ot_version(void) { return "0.1.0 gfx950"; }
