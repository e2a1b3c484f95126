// Error reporting and argument validation shared by every C entry point.
#include <stdarg.h>
#include <stdio.h>

#include "common.hpp"

namespace fm {

static thread_local char g_err[512] = "";

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return code;
}

void clear_error() { g_err[0] = '\0'; }

int need(const void* p, const char* name) {
  if (!p) return fail(MOE_ERR_ARG, "%s must not be NULL", name);
  return MOE_OK;
}

int need_aligned(const void* p, const char* name) {
  if (p && !aligned16(p)) return fail(MOE_ERR_ALIGN, "%s is not 16-byte aligned", name);
  return MOE_OK;
}

int need_dtype_float(int dtype, const char* name) {
  if (dtype != MOE_F32 && dtype != MOE_BF16)
    return fail(MOE_ERR_UNSUPPORTED, "%s=%d: expected MOE_F32 or MOE_BF16", name, dtype);
  return MOE_OK;
}

int check_launch(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(MOE_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return MOE_OK;
}

}  // namespace fm

extern "C" const char* moe_last_error(void) { return fm::g_err; }
extern "C" int moe_abi_version(void) { return FLUXMOE_ABI_VERSION; }
