// The thread-local error message of the C ABI (fcg_last_error), shared by the
// library's host translation units.
#pragma once

#include <string>

#include "fcg.h"

namespace fcg {
// Record msg as the calling thread's last error and return s.
fcg_status report(fcg_status s, const std::string& msg);
}  // namespace fcg
