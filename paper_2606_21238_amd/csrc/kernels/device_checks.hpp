// Device checks of the kernel sources (included by each .hip file once; see internal.hpp).
// With ARCKV_DEVICE_CHECKS, every source gets its own per-device word pair `g_checks` (code
// bits, occurrences) and a reader; otherwise the record macros compile to nothing.  Records
// are vector atomics on global memory; nothing traps.
#pragma once

#include <hip/hip_runtime.h>

#include "../host/internal.hpp"

#ifdef ARCKV_DEVICE_CHECKS
namespace {
__device__ unsigned int g_checks[2];
}
// every lane whose condition holds records once
#define ARCKV_CHECK_LANE(cond, code)               \
  do {                                             \
    if (cond) {                                    \
      atomicOr(&g_checks[0], (code));              \
      atomicAdd(&g_checks[1], 1u);                 \
    }                                              \
  } while (0)
// a wave-uniform condition: lane 0 of the wave records once
#define ARCKV_CHECK_WAVE(cond, code) ARCKV_CHECK_LANE((cond) && (threadIdx.x & 63) == 0, code)

#define ARCKV_DEFINE_CHECK_READER(fn)                                                           \
  int32_t arckv::fn(void* stream, bool reset, uint32_t* bits, uint32_t* count) {                \
    auto* s = static_cast<hipStream_t>(stream);                                                 \
    void* p = nullptr;                                                                           \
    uint32_t host[2] = {0, 0};                                                                   \
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(g_checks)) != hipSuccess ||                           \
        hipMemcpyAsync(host, p, sizeof(host), hipMemcpyDeviceToHost, s) != hipSuccess ||         \
        hipStreamSynchronize(s) != hipSuccess)                                                    \
      return arckv::fail(ARCKV_EDEVICE, "device checks: reading the record failed");            \
    if (reset && (hipMemsetAsync(p, 0, sizeof(host), s) != hipSuccess ||                          \
                  hipStreamSynchronize(s) != hipSuccess))                                         \
      return arckv::fail(ARCKV_EDEVICE, "device checks: clearing the record failed");           \
    *bits = host[0];                                                                             \
    *count = host[1];                                                                            \
    return ARCKV_OK;                                                                             \
  }
#else
#define ARCKV_CHECK_LANE(cond, code) do { } while (0)
#define ARCKV_CHECK_WAVE(cond, code) do { } while (0)
#define ARCKV_DEFINE_CHECK_READER(fn)                                                           \
  int32_t arckv::fn(void*, bool, uint32_t*, uint32_t*) {                                         \
    return arckv::fail(ARCKV_EUNSUPPORTED, "device checks: the library was built without them");  \
  }
#endif
