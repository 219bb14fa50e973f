#include "errors.hpp"

namespace tp {
std::string& last_error() {
  thread_local std::string msg;
  return msg;
}
}  // namespace tp

extern "C" const char* tp_last_error(void) { return tp::last_error().c_str(); }
