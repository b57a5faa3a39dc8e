// Status strings and the thread-local message behind bros_last_error().
#include "bros_attn.h"
#include "bros_error.h"

#include <cstdarg>
#include <cstdio>
#include <string>

namespace {
thread_local std::string g_last_error;
}

namespace bros {

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

int ok() {
  g_last_error.clear();
  return BROS_OK;
}

}  // namespace bros

extern "C" {

const char* bros_status_str(int status) {
  switch (status) {
    case BROS_OK: return "BROS_OK";
    case BROS_E_NULL: return "BROS_E_NULL";
    case BROS_E_SHAPE: return "BROS_E_SHAPE";
    case BROS_E_DTYPE: return "BROS_E_DTYPE";
    case BROS_E_UNSUPPORTED: return "BROS_E_UNSUPPORTED";
    case BROS_E_WORKSPACE: return "BROS_E_WORKSPACE";
    case BROS_E_HIP: return "BROS_E_HIP";
    case BROS_E_TABLE: return "BROS_E_TABLE";
    case BROS_E_NOMEM: return "BROS_E_NOMEM";
    default: return "BROS_E_UNKNOWN";
  }
}

const char* bros_last_error(void) { return g_last_error.c_str(); }

int bros_abi_version(void) { return 9; }

}  // extern "C"
