// Status strings and the thread-local error detail.
#include <stdarg.h>
#include <stdio.h>

#include "oda_internal.h"

namespace {
thread_local char g_last_error[512] = "";
}

namespace oda {

oda_status fail(oda_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return s;
}

oda_status ok() {
  g_last_error[0] = '\0';
  return ODA_OK;
}

}  // namespace oda

extern "C" const char* oda_status_string(oda_status status) {
  switch (status) {
    case ODA_OK: return "ODA_OK";
    case ODA_ERR_NULL: return "ODA_ERR_NULL: a required pointer is NULL";
    case ODA_ERR_SHAPE: return "ODA_ERR_SHAPE: inconsistent or out-of-range sizes";
    case ODA_ERR_UNSUPPORTED: return "ODA_ERR_UNSUPPORTED: valid but not implemented";
    case ODA_ERR_WORKSPACE: return "ODA_ERR_WORKSPACE: workspace missing or too small";
    case ODA_ERR_HIP: return "ODA_ERR_HIP: a HIP launch failed";
  }
  return "unknown oda_status";
}

extern "C" const char* oda_last_error(void) { return g_last_error; }
