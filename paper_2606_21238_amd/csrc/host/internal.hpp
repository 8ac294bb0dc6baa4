// Internal declarations shared by the host-side translation units of libarckv.
#pragma once

#include <cstdarg>
#include <cstdint>
#include <string>

#include "arckv.h"

namespace arckv {

// Query columns (token x query head of one KV group) per attention work-group: kTileWaves
// wave64s, each owning kWaveCols columns.  Shared by the host work plan and the kernel.
constexpr int kWaveCols = 32;
constexpr int kTileWaves = 8;
constexpr int kTileCols = kTileWaves * kWaveCols;

// Records a thread-local message for arckv_last_error() and returns `code`.
int32_t fail(int32_t code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();

}  // namespace arckv
