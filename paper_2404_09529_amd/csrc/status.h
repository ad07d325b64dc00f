// Thread-local error text behind pp_last_error(), and the argument checks shared by the
// entry points.
#pragma once
#include "prepack.h"

namespace pp {
void clear_error();
pp_status fail(pp_status code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
// Sizes, dtype and the shape limits of the kernels (the errors pp_prefill documents).
pp_status validate_config(const pp_config* c);
// Every weight pointer of every layer non-NULL.
pp_status validate_weights(const pp_config* c, const pp_weights* w);
}  // namespace pp
