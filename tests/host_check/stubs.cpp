// Kernel launchers replaced by stubs that report "no device": the host
// sanitizer build of the C ABI (api.cpp) links these instead of the HIP
// kernels, so that every host path -- argument checks, workspace layout,
// launch decisions, profiling bookkeeping -- runs on a machine without a GPU.
#include "prefill.h"

namespace hagdn {
hipError_t launch_chunk_index(const PrefillArgs &, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_chunk_local(const PrefillArgs &, bool, bool, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_state_prop(const PrefillArgs &, bool, bool, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_overlap_setup(const PrefillArgs &, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_overlapped(const PrefillArgs &, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_state_walk(const PrefillArgs &, bool, int, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_seg_maps(const PrefillArgs &, bool, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_seg_transfer(const PrefillArgs &, bool, bool, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_seg_state(const PrefillArgs &, bool, bool, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_decode(const DecodeArgs &, bool, bool, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_copy(const void *, void *, size_t, int, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_mfma_loop(int, int, float *, hipStream_t) { return hipErrorNoDevice; }
}  // namespace hagdn
