// Host-only stand-ins for the kernel launchers of the HIP library, for the
// sanitizer build of the host code (pda_host.cpp compiled by the host C++
// compiler with AddressSanitizer and UndefinedBehaviorSanitizer). The host
// tests that run against that build stop at argument validation, before any
// launch; reaching one of these is reported as a launch failure.
#include "pda_internal.h"

namespace pda {

hipError_t launch_decode(const DecodeArgs&, Variant, KvType, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_combine(const DecodeArgs&, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_prefix(const DecodeArgs&, int, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_append(const AppendArgs&, KvType, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_prefill(const PrefillArgs&, KvType, hipStream_t) { return hipErrorInvalidValue; }
hipError_t decode_occupancy(Variant, KvType, int, int, bool, int* w) {
  *w = 1;
  return hipErrorInvalidValue;
}
hipError_t scratch_address(void** p) {
  *p = nullptr;
  return hipErrorInvalidValue;
}

}  // namespace pda
