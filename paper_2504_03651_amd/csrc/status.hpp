// status.hpp -- the calling thread's error detail behind echo_last_error().
#pragma once

namespace echo {

// Records a printf-style detail for echo_last_error() and returns `code`.
int fail(int code, const char *fmt, ...);
// Clears the calling thread's detail (every entry point starts with it).
void clear_error();
// Whether echo_profile(1) is on for the calling thread.
bool profile_enabled();

}  // namespace echo
