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
// Narrow plans give every work-group a list of this many work items (its items in order, then
// idle padding): the attention launch has n_work / kListItems work-groups.
constexpr int kListItems = 8;

// Whether the cache was created in check mode (block digests verified by every plan).
bool cache_checks_blocks(const arckv_cache* c);

// Device checks (a build with ARCKV_DEVICE_CHECKS defined): a kernel that clamps or skips an
// out-of-range index also records it in a per-device word pair of its source file (bits OR-ed,
// occurrences counted).  Each kernel source provides a reader: it waits for `stream`, reads
// the pair of the current device and, if reset, clears it.  Without device checks they return
// ARCKV_EUNSUPPORTED.
int32_t read_scatter_checks(void* stream, bool reset, uint32_t* bits, uint32_t* count);
int32_t read_attention_checks(void* stream, bool reset, uint32_t* bits, uint32_t* count);

// Records a thread-local message for arckv_last_error() and returns `code`.
int32_t fail(int32_t code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();

}  // namespace arckv
