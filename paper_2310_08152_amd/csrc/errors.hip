// Host-side error reporting shared by every entry point of libsckv.so.
#include <string>

#include "sckv_common.h"

namespace sckv {

static thread_local std::string g_last_error;

void set_error(const std::string& msg) { g_last_error = msg; }
void clear_error() { g_last_error.clear(); }

int fail(int code, const std::string& msg) {
  g_last_error = msg;
  return code;
}

int hip_check(hipError_t e, const char* what) {
  if (e == hipSuccess) return SCKV_OK;
  g_last_error = std::string(what) + ": " + hipGetErrorString(e);
  return SCKV_EHIP;
}

}  // namespace sckv

extern "C" const char* sckv_last_error(void) { return sckv::g_last_error.c_str(); }

extern "C" const char* sckv_version(void) { return "sckv 0.1 (gfx950)"; }
