// Thread-local error message shared by the C ABI entry points.
#pragma once

namespace bros {
// Record a formatted message for bros_last_error() and return `code`.
int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
// Clear the message and return BROS_OK.
int ok();
}  // namespace bros
