#include "ra_error.h"

namespace {
thread_local std::string g_last_error;
}

int ra_fail(int code, const std::string& msg) {
  g_last_error = msg;
  return code;
}

int ra_ok() { return RA_OK; }

extern "C" const char* ra_last_error(void) { return g_last_error.c_str(); }
