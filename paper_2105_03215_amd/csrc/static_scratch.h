// Static per-device scratch used as the arena of allocation-free runs.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace byoc {

// Bytes of the static scratch array every GPU holds (64 MiB).
constexpr int64_t kStaticScratchBytes = int64_t(64) << 20;

// Device address of `device`'s copy of the array, looked up on the first
// call for that device and cached; later calls only read the table.
hipError_t static_scratch_ptr(int device, void** ptr);

}  // namespace byoc
