// Thread-local last-error reporting shared by the library's C entry points.
#pragma once

namespace optimus {

// Record a printf-style message for enc_last_error() and return `code`.
int set_error(int code, const char *fmt, ...);
// Clear the message and return ENC_OK.
int clear_error();

}  // namespace optimus
