// status.cpp -- the decode library's per-thread last-error message (status.h).
// Plain host C++, shared by every entry point of libapex_decode.so.
#include <stdarg.h>
#include <stdio.h>

#include "status.h"

namespace apex {

namespace {
thread_local char g_last_error[512] = "";
}

int fail(int code, const char* fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
    va_end(ap);
    return code;
}

void clear_error() { g_last_error[0] = 0; }

const char* last_error_message() { return g_last_error; }

}  // namespace apex
