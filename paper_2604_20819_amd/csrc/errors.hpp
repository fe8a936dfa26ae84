// Thread-local error text behind cqsa_last_error().
#pragma once

#include <string>

#include "cqsa.h"

namespace cqsa {

std::string& error_slot();

inline void clear_error() { error_slot().clear(); }

inline cqsa_status fail(cqsa_status s, const std::string& msg) {
  error_slot() = msg;
  return s;
}

inline const char* last_error_cstr() { return error_slot().c_str(); }

}  // namespace cqsa
