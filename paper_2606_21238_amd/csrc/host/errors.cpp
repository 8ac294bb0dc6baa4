// Thread-local error messages and small ABI queries of libarckv.
#include <cstdio>

#include "internal.hpp"

namespace {
thread_local char g_msg[512] = "";
}

namespace arckv {

int32_t fail(int32_t code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(g_msg, sizeof(g_msg), fmt, ap);
  va_end(ap);
  return code;
}

void clear_error() { g_msg[0] = '\0'; }

}  // namespace arckv

extern "C" const char* arckv_last_error(void) { return g_msg; }

extern "C" int32_t arckv_version(void) { return 1; }

extern "C" int64_t arckv_pool_bytes(int64_t num_blocks, int32_t num_kv_heads, int32_t head_dim) {
  if (num_blocks < 0 || num_kv_heads < 1 || head_dim < 1) return -1;
  return num_blocks * num_kv_heads * ARCKV_BLOCK_TOKENS * static_cast<int64_t>(head_dim) * 2;
}
