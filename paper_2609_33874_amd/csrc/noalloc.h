// Per-device fixed scratch of the allocation-free scoring entry point.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>

#include "../../include/jet.h"

namespace jet {

constexpr size_t kNoallocScratchBytes = (size_t)JET_NOALLOC_SCRATCH_BYTES;
constexpr int kNoallocMaxDevices = 64;

// Looks up the device address of the scratch array on `device`, which must be
// the current device; once per device (later calls return at once).
hipError_t noalloc_scratch_init(int device);
// The address found by noalloc_scratch_init for `device`, or NULL.
void *noalloc_scratch(int device);

}  // namespace jet
