// Thread-local error reporting of the C ABI.
#include <string>

#include "internal.hpp"

namespace tbias {

namespace {
thread_local std::string g_err;
}

void set_error(const std::string& msg) { g_err = msg; }

int fail(int code, const std::string& msg) {
  g_err = msg;
  return code;
}

}  // namespace tbias

extern "C" const char* tb_last_error(void) { return tbias::g_err.c_str(); }
