// The library's own device scratch for callers that cannot allocate (see
// comem_decode_attn_noalloc): a file-scope device array, one copy per GPU,
// kept until the process ends.
//
// Host code never passes the array's name to a kernel or a runtime call: in
// host code that name is a host-side stand-in, not a device address. The
// device address of each GPU's copy is looked up once, with that GPU
// current, by hipGetSymbolAddress in scratch_setup (called by
// comem_decode_attn_init for a real device) and kept per device; every later
// use goes through that pointer.
//
// Layout: the first kScratchTicketBytes hold ticket and work-queue counters
// (zero between calls: filled with zeros at set-up, and every kernel returns
// the counters it takes to zero before it ends), the rest the split partial
// results, which a call always writes before it reads them. Because the
// counter region has a fixed place whatever the plan, a call of one plan
// never finds another plan's partial results where it expects zeros.
#include <hip/hip_runtime.h>

#include <cstddef>
#include <mutex>

#include "comem_decode_attn.h"
#include "noalloc.h"

namespace comem {
namespace {

__device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_mutex;
void* g_ptr[kScratchMaxDevices];  // device address of `scratch` on each device (nullptr: not set up)

}  // namespace

bool scratch_setup(int device) {
  if (device < 0 || device >= kScratchMaxDevices) return false;
  std::lock_guard<std::mutex> lock(g_mutex);
  if (g_ptr[device] != nullptr) return true;
  int prev = -1;
  if (hipGetDevice(&prev) != hipSuccess) return false;
  if (prev != device && hipSetDevice(device) != hipSuccess) return false;
  void* ptr = nullptr;
  hipError_t err = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
  if (err == hipSuccess && ptr == nullptr) err = hipErrorInvalidSymbol;
  // The counter region must start at zero; set-up runs outside any stream
  // capture, so a synchronous fill is fine here.
  if (err == hipSuccess) err = hipMemset(ptr, 0, kScratchTicketBytes);
  if (err == hipSuccess) err = hipDeviceSynchronize();
  if (prev != device) (void)hipSetDevice(prev);
  if (err != hipSuccess) return false;
  g_ptr[device] = ptr;
  return true;
}

void* scratch_pointer(int device) {
  if (device < 0 || device >= kScratchMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_mutex);
  return g_ptr[device];
}

}  // namespace comem
