// Status strings and the thread-local error message of the C ABI.
#include <cstdarg>
#include <cstdio>

#include "kernels.h"

namespace catq {

static thread_local char g_msg[512] = "";

void set_error(const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(g_msg, sizeof(g_msg), fmt, ap);
  va_end(ap);
}

void clear_error() { g_msg[0] = '\0'; }

}  // namespace catq

extern "C" const char* catq_status_string(catq_status s) {
  switch ((int)s) {
    case CATQ_OK: return "CATQ_OK";
    case CATQ_ERR_NULL: return "CATQ_ERR_NULL";
    case CATQ_ERR_SHAPE: return "CATQ_ERR_SHAPE";
    case CATQ_ERR_DTYPE: return "CATQ_ERR_DTYPE";
    case CATQ_ERR_VALUE: return "CATQ_ERR_VALUE";
    case CATQ_ERR_ALIGN: return "CATQ_ERR_ALIGN";
    case CATQ_ERR_WORKSPACE: return "CATQ_ERR_WORKSPACE";
    case CATQ_ERR_HIP: return "CATQ_ERR_HIP";
  }
  return "CATQ_ERR_UNKNOWN";
}

extern "C" const char* catq_last_error_message(void) { return catq::g_msg; }
