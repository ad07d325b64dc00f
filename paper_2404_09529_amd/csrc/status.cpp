#include "status.h"

#include <cstdarg>
#include <cstdio>

namespace {
thread_local char g_msg[512] = "";
}

namespace pp {
void clear_error() { g_msg[0] = '\0'; }

pp_status fail(pp_status code, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(g_msg, sizeof g_msg, fmt, ap);
    va_end(ap);
    return code;
}
}  // namespace pp

extern "C" const char* pp_last_error(void) { return g_msg; }

extern "C" const char* pp_version(void) { return "0.1.0 gfx950"; }
