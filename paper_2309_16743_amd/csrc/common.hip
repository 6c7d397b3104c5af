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

}  // namespace ot

extern "C" const char* ot_last_error(void) { return ot::t_error.c_str(); }

extern "C" const char* ot_version(void) { return "0.1.0 gfx950"; }
