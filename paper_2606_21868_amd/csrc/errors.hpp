// The thread's last-error message of the C ABI (wisp_last_error), shared by the library's sources.
#pragma once

#include <string>

#include "wisp.h"

namespace wisp {
wisp_status set_error(wisp_status s, const std::string& msg);   // records msg, returns s
}  // namespace wisp
