// Status strings and the thread-local error message.
#include <cstdarg>
#include <cstdio>

#include "gnnshap.h"

namespace gnnshap {

static thread_local char g_msg[512] = "";

int fail(int status, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_msg, sizeof(g_msg), fmt, ap);
  va_end(ap);
  return status;
}

void clear_error() { g_msg[0] = '\0'; }

}  // namespace gnnshap

extern "C" {

const char* gnnshap_status_str(int status) {
  switch (status) {
    case GNNSHAP_OK: return "ok";
    case GNNSHAP_EINVAL: return "invalid argument";
    case GNNSHAP_ECAPACITY: return "buffer or workspace too small";
    case GNNSHAP_EHIP: return "HIP runtime error";
    case GNNSHAP_ESINGULAR: return "singular system";
    case GNNSHAP_EUNSUPPORTED: return "unsupported";
    default: return "unknown status";
  }
}

const char* gnnshap_last_error(void) { return gnnshap::g_msg; }

int gnnshap_version(void) { return 100; /* 0.1.0 */ }

}  // extern "C"
