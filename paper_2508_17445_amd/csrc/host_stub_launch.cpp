// Host-only stand-ins for the kernel launchers, for the sanitizer build of the
// host core (node table, planner, C-ABI bookkeeping).  Every launch reports
// that no device is present; the metadata, validation and error paths under
// test never launch.
#include "kernels.h"

namespace treepo {

hipError_t launch_partial(const DecodeArgs&, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_combine(const DecodeArgs&, hipStream_t) { return hipErrorNoDevice; }
int32_t partial_workgroups_per_cu() { return 2; }
hipError_t noalloc_scratch(void**, uint64_t**) { return hipErrorNoDevice; }
hipError_t launch_advantage(const AdvantageArgs&, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_prefill(const PrefillArgs&, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_kv_append_dev(const uint16_t*, const uint16_t*, uint16_t*, uint16_t*, int64_t, int32_t, int32_t,
                                const AppendPiece*, int32_t, const int2*, int32_t, int32_t*, hipStream_t) {
  return hipErrorNoDevice;
}
hipError_t launch_kv_append(const uint16_t*, const uint16_t*, uint16_t*, uint16_t*, int64_t, int32_t, int32_t,
                            const AppendPiece*, int32_t, const int32_t*, const int32_t*, int32_t, int32_t*,
                            hipStream_t) {
  return hipErrorNoDevice;
}

}  // namespace treepo
