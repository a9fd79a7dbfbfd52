// Status strings, the thread-local error message and launch checking for the C ABI.
#include "fl_common.h"

#include <cstring>

namespace fl {

static thread_local char g_last_error[512] = "";

int set_error(int status, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return status;
}

int check_launch(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess)
    return set_error(FL_E_HIP, "%s: launch failed: %s", what, hipGetErrorString(e));
  return FL_OK;
}

}  // namespace fl

extern "C" const char* fl_status_str(int status) {
  switch (status) {
    case FL_OK: return "FL_OK";
    case FL_E_NULL: return "FL_E_NULL: a required pointer is NULL";
    case FL_E_SHAPE: return "FL_E_SHAPE: inconsistent or unsupported sizes";
    case FL_E_RANGE: return "FL_E_RANGE: a count is out of range";
    case FL_E_UNSUPPORTED: return "FL_E_UNSUPPORTED: unsupported bit width, axis, mode or flag";
    case FL_E_WORKSPACE: return "FL_E_WORKSPACE: workspace missing or too small";
    case FL_E_HIP: return "FL_E_HIP: the HIP runtime rejected a launch";
    case FL_E_INTERNAL: return "FL_E_INTERNAL: internal error";
    default: return "unknown status";
  }
}

extern "C" const char* fl_last_error(void) { return fl::g_last_error; }

extern "C" int fl_abi_version(void) { return FL_ABI_VERSION; }
