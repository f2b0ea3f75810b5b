// Error reporting and version of the C ABI.
#include "nsd_internal.h"

namespace nsd {
static thread_local char g_err[512] = "no error";

void set_error(const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
}
}  // namespace nsd

extern "C" int32_t nsd_version(void) { return (0 << 16) | 1; }
extern "C" const char* nsd_last_error(void) { return nsd::g_err; }
