// Internal interface of the library-owned device scratch (noalloc.hip).
#pragma once

#include <cstddef>

#include "comem_decode_attn.h"

namespace comem {

constexpr std::size_t kScratchBytes = COMEM_NOALLOC_SCRATCH_BYTES;   // per GPU, held until the process ends
constexpr std::size_t kScratchTicketBytes = 64 * 1024;               // counters at the start of the scratch
constexpr int kScratchMaxDevices = 64;

// Look up this device's copy of the scratch array (with the device current)
// and fill its counter region with zeros; once per device, thread-safe.
// Returns false on a HIP error or a device ordinal outside [0, 64).
bool scratch_setup(int device);

// The device address scratch_setup found, or nullptr if it did not succeed.
void* scratch_pointer(int device);

}  // namespace comem
