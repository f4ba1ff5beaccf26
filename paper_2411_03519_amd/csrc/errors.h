// Error reporting shared by the library's translation units: the message of
// the last failed call on this thread, returned by metro_last_error().
#pragma once

#include "../../include/metro.h"

namespace metro {

// Record a printf-style message and return st.
metro_status report(metro_status st, const char* fmt, ...);
// Forget the last message (every entry point starts with this).
void clear_error();

}  // namespace metro
