// Error reporting shared by the C-ABI translation units.
#pragma once

namespace kvattn {

// Record a printf-style message as the calling thread's last error; returns code.
int set_error(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();

}  // namespace kvattn
