// Shared by the library's sources; not part of the C ABI.
#pragma once

namespace eb_detail {

// Record a printf-style message as the calling thread's last error
// (eb_last_error) and return code.  The message goes into a fixed
// thread-local buffer (truncated if longer): no allocation, no exception.
int fail(int code, const char *fmt, ...) __attribute__((format(printf, 2, 3)));

// The calling thread's last message ("" if none).
const char *last_error();

// What an entry point returns when something below it threw (its own paths
// allocate nothing, so only a runtime library could): EB_ERR_NOMEM.
int unexpected_exception(const char *who);

} // namespace eb_detail
