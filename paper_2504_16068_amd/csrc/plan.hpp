// The plan object behind the opaque allegro_tp_plan handle (host side).
#pragma once

#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <string>

#include "cg_builder.hpp"

struct allegro_tp_plan {
  int lmax = 0, U = 0, flags = 0;
  allegro::TPTable table;
  int *status = nullptr;  // device word for ALLEGRO_VALIDATE
  std::mutex validate_mu;
  // polls before a wait between the waves of the matrix-core backward gives
  // up (0 only to test that path: every such wait then gives up at once)
  int spin_limit = 1 << 24;
};

namespace allegro_internal {

// Thread-local message of the last failed call, shared by every translation
// unit of the library; fail() sets it and returns code.
inline std::string &last_error_slot() {
  thread_local std::string msg;
  return msg;
}

inline const char *last_error() { return last_error_slot().c_str(); }

inline int fail(int code, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  last_error_slot() = buf;
  return code;
}

}  // namespace allegro_internal
