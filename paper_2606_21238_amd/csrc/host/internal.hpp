// Internal declarations shared by the host-side translation units of libarckv.
#pragma once

#include <cstdarg>
#include <cstdint>
#include <string>

#include "arckv.h"

namespace arckv {

// Query columns (token x query head of one KV group) per attention work-group: each wave64
// owns kWaveCols columns; a work-group has 8 waves (wide tiles) or 4 waves (narrow tiles, for
// batches whose suffixes are short).  Shared by the host work plan and the kernel.
constexpr int kWaveCols = 32;
constexpr int kWideCols = 8 * kWaveCols;
constexpr int kNarrowCols = 4 * kWaveCols;

// Records a thread-local message for arckv_last_error() and returns `code`.
int32_t fail(int32_t code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();

}  // namespace arckv
