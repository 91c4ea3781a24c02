// log.hpp -- opt-in call logging for the C ABI.
//
// With the environment variable QG_LOG set to anything but "" or "0" when
// the library is first used, every entry point writes one line to stderr:
// its name, its scalar arguments and the status it returns (with the HIP
// error for QG_ERR_HIP). Off by default; the check is one cached flag.
#pragma once
#include <cstdlib>

#include "qgemm.h"

namespace qg {

inline bool log_enabled() {
  static const bool on = [] {
    const char* v = std::getenv("QG_LOG");
    return v != nullptr && v[0] != '\0' && !(v[0] == '0' && v[1] == '\0');
  }();
  return on;
}

void log_call(const char* fn, qg_status st, const char* fmt, ...) __attribute__((format(printf, 3, 4)));

}  // namespace qg
