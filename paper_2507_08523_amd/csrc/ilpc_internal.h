// Internal helpers shared by the library's translation units (not part of the ABI).
#pragma once

#include <cstdarg>

namespace ilpc {

// Records a message for ilpc_last_error() on the calling thread and returns `code`.
int set_error(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));

}  // namespace ilpc
