// Internal helpers shared by the host-side translation units of librip.
#pragma once

#include <cstdint>
#include <functional>

#include "rip.h"

namespace rip {

// Records a printf-style message as the calling thread's last error and
// returns `code`, so that error paths read `return fail(RIP_E_INVAL, ...)`.
int32_t fail(int32_t code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();

// Number of workers of a scheduler.
int32_t sched_workers(const rip_sched* s);

// Group generation for `step` (as rip_schedule_groups), then `then()`; the
// scheduler keeps the new state only if both return RIP_OK, else it is left
// exactly as it was.
int32_t schedule_then(rip_sched* s, int64_t step, const uint8_t* eligible, int32_t* active,
                      int32_t* n_active, int32_t* group_offsets, int32_t* members,
                      int32_t* n_groups, const std::function<int32_t()>& then);

}  // namespace rip
