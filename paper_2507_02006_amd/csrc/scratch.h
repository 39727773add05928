// Fixed per-device workspace of the allocation-free entry point.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace aires {

// Bytes of the workspace array each device holds (64 MiB).
constexpr int64_t kScratchBytes = int64_t(64) << 20;

// Device address of the current device's workspace array, looked up once
// per device (hipGetSymbolAddress) and cached; hipSuccess or the error.
hipError_t scratch_address(void** out);

}  // namespace aires
