// Fixed device workspace of pda_paged_decode_attention_noalloc (include/pda.h):
// the decode step's partial results, per-sequence prefix sums, chunk counter
// and status word, in the layout of the stream workspaces of the allocating
// entry points, for callers that cannot allocate device memory.

#include "pda_internal.h"

namespace pda {

// Zero at load (static storage duration), one copy per device, shared by
// every call on that device until the process ends. In host code this name
// denotes a host-side stand-in, not device memory: host code never passes it
// to a kernel or a copy, only the address scratch_address() returns.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

// The current device's copy of the array (the caller makes the device
// current and keeps the address per device).
hipError_t scratch_address(void** ptr) {
  *ptr = nullptr;
  return hipGetSymbolAddress(ptr, HIP_SYMBOL(scratch));
}

}  // namespace pda
