// Status and error text shared by the C ABI sources of librksc.
#pragma once

#include <string>

#include "../../include/rksc.h"

namespace rksc {

// The calling thread's last error text (what rksc_last_error returns).
std::string& last_error();
// Records the formatted message and returns st.
rksc_status fail(rksc_status st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
// Clears the message and returns RKSC_OK.
rksc_status ok();

}  // namespace rksc
