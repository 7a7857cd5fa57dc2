// Thread-local error message behind lssvm_last_error(), shared by the
// training path and the host IO routines.
#pragma once

namespace lssvm {

// Record a printf-style message for lssvm_last_error() and return `code`.
int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));

// Forget the last message (each entry point starts with an empty one).
void clear_error();

}  // namespace lssvm
