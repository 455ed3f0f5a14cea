// The library-owned device scratch of mssa_attention_noalloc (noalloc.hip).
#pragma once

#include <hip/hip_runtime_api.h>

#include <cstdint>

namespace mssa {

// Bytes of the scratch array each device holds (MSSA_NOALLOC_SCRATCH_BYTES).
constexpr int64_t kScratchBytes = int64_t{256} << 20;

// Device address of the current device's scratch array: looked up with
// hipGetSymbolAddress on the first call on that device (the device current),
// then kept.  Thread-safe.
hipError_t scratch_address(void** out);

}  // namespace mssa
