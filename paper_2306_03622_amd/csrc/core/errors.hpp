// Thread-local error message behind tp_last_error().
#pragma once
#include <string>

#include "torpor.h"

namespace tp {
std::string& last_error();
inline tp_status fail(tp_status s, const std::string& msg) {
  last_error() = msg;
  return s;
}
inline tp_status ok() {
  last_error().clear();
  return TP_OK;
}
}  // namespace tp
