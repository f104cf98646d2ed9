// Per-thread error message shared by every entry point of the library
// (returned by cs_last_error()).  Host-only: no HIP types.
#pragma once

namespace cs {

// Record a printf-style message for the calling thread and return `status`.
int fail(int status, const char* fmt, ...) __attribute__((format(printf, 2, 3)));

// Clear the calling thread's message and return CS_OK.
int ok();

}  // namespace cs
