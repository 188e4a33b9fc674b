// Shared by the library's sources; not part of the C ABI.
#pragma once

#include <string>

namespace eb_detail {

// Record msg as the calling thread's last error (eb_last_error) and return code.
int fail(int code, const std::string &msg);

} // namespace eb_detail
