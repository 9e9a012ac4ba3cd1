// Internal helpers shared by the translation units of libonexn.so.
#pragma once

#include <cstdarg>
#include <cstdint>

#include "onexn.h"

namespace onexn {

// Records a printf-style message for onexn_last_error() and returns `s`.
onexn_status fail(onexn_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));

// Clears the calling thread's last error message.
void clear_error();

}  // namespace onexn
