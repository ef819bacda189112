// Internal helpers shared by the host-side translation units of libdcp.
#pragma once

#include <cstdarg>
#include <cstdint>

#include "dcp.h"

namespace dcp {

// Records a printf-style message as the calling thread's last error and
// returns `code`, so call sites can write `return fail(DCP_ERR_..., ...)`.
int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));

// Clears the calling thread's last error message.
void clear_error();

}  // namespace dcp
