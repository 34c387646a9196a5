// status.h -- error reporting shared by the library's entry points.
//
// Every extern "C" entry point returns an apex_status and, on failure, leaves
// a message for apex_decode_last_error() (one buffer per host thread).
#pragma once

namespace apex {

// Stores the formatted message as the calling thread's last error and returns code.
__attribute__((visibility("hidden"), format(printf, 2, 3))) int fail(int code, const char* fmt, ...);

// Clears the calling thread's last error (entry points call it first).
__attribute__((visibility("hidden"))) void clear_error();

// The calling thread's last error ("" if none).
__attribute__((visibility("hidden"))) const char* last_error_message();

}  // namespace apex
