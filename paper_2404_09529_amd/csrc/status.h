// Thread-local error text behind pp_last_error().
#pragma once
#include "prepack.h"

namespace pp {
void clear_error();
pp_status fail(pp_status code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
}  // namespace pp
