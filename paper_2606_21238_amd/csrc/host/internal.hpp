// Internal declarations shared by the host-side translation units of libarckv.
#pragma once

#include <cstdarg>
#include <cstdint>
#include <string>

#include "arckv.h"

namespace arckv {

// Query columns (token x query head of one KV group) per attention work-group, shared by the
// host work plan and the kernel: wide tiles (8 waves x 32 columns) and narrow tiles for short
// suffixes and decode-like batches (4 x 32 columns, the 8 waves split over the keys of each
// K/V tile).
constexpr int kWaveCols = 32;
constexpr int kWideCols = 8 * kWaveCols;
constexpr int kNarrowCols = 4 * kWaveCols;
// Longest key range of one attention work item: longer ranges are split into pieces (merged by
// the combine), so that the item's block-table entries (kMaxItemKeys / 16) fit in LDS.
constexpr int kMaxItemKeys = 65536;

// Whether the cache was created in check mode (block digests verified by every plan).
bool cache_checks_blocks(const arckv_cache* c);

// Records a thread-local message for arckv_last_error() and returns `code`.
int32_t fail(int32_t code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();

}  // namespace arckv
