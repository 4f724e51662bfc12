// Error reporting shared by the C-ABI sources: a failing entry point records its reason
// (read back with s2l_last_error) and returns the status; a succeeding one clears it.
#pragma once
#include "s2l.h"

namespace s2l {

s2l_status fail(s2l_status st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
s2l_status ok();

}  // namespace s2l
