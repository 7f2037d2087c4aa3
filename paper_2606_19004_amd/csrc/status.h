// Error reporting shared by the library's translation units: sets the thread-local message
// returned by dit_last_error_message() and passes the status through.
#pragma once
#include "../../include/ditstep.h"

namespace dit {
dit_status set_error(dit_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
}
