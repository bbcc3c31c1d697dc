// Status codes and the thread-local error message behind kvp_last_error().
#pragma once

#include <cstdarg>
#include <cstdio>

#include "kvpipe.h"

namespace kvp {

char* last_error_buffer();   // thread-local, 512 bytes

inline int fail(int code, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(last_error_buffer(), 512, fmt, ap);
    va_end(ap);
    return code;
}

inline int ok() { return KVP_OK; }

}  // namespace kvp
