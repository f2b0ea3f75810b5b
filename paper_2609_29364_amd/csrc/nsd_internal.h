// Internal helpers shared by the library's translation units (not installed).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdio.h>
#include <stdarg.h>
#include "nebulasd.h"

namespace nsd {

// Thread-local message for the last non-OK status (nsd_last_error).
void set_error(const char* fmt, ...);

inline nsd_status fail(nsd_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  set_error("%s", buf);
  return st;
}

// Status of the launch just enqueued.
inline nsd_status check_launch(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(NSD_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return NSD_OK;
}

// Clear an error left by an earlier unrelated call so check_launch reports ours.
inline void clear_stale_error() { (void)hipGetLastError(); }

}  // namespace nsd
