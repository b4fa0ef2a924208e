// Internal helpers shared by the host-side translation units of librip.
#pragma once

#include <cstdint>

#include "rip.h"

namespace rip {

// Records a printf-style message as the calling thread's last error and
// returns `code`, so that error paths read `return fail(RIP_E_INVAL, ...)`.
int32_t fail(int32_t code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();

}  // namespace rip
