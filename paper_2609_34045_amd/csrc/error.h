// Thread-local error message behind kf_last_error(), shared by every C-ABI entry point.
#pragma once
#include "kafila_stage.h"

namespace kf {
// Records the message for kf_last_error() and returns `code`.
kf_status fail(kf_status code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
// Empties the message (after a call that succeeds where an earlier one failed).
void clear_error();
}  // namespace kf
