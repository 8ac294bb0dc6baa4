// Internal declarations shared by the host-side translation units of libarckv.
#pragma once

#include <cstdarg>
#include <cstdint>
#include <string>

#include "arckv.h"

namespace arckv {

// Records a thread-local message for arckv_last_error() and returns `code`.
int32_t fail(int32_t code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();

}  // namespace arckv
