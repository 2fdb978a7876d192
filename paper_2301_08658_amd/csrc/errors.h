// Internal: the library's per-thread last-error message (read back by
// atp_last_error()).
#pragma once

#include "../../include/atp.h"

namespace atp {
// Records a printf-style message as the calling thread's last error and
// returns `s`.
atp_status set_error(atp_status s, const char* fmt, ...);
}  // namespace atp
