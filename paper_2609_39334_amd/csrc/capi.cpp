// Error reporting shared by every C entry point: a thread-local message behind tkv_last_error().
#include <cstdarg>
#include <cstdio>
#include <string>

#include "internal.h"

namespace {
thread_local std::string g_error;
}

namespace tkv {

int set_error(int code, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_error = buf;
    return code;
}

void clear_error() { g_error.clear(); }

}  // namespace tkv

TKV_EXPORT const char* tkv_last_error(void) { return g_error.c_str(); }
