// Host-only stand-ins for the kernel launchers of the attention library, for
// the sanitizer build of its C-ABI front end (api.cpp): the validation,
// workspace sizing and dispatch logic run under AddressSanitizer and
// UndefinedBehaviorSanitizer on the CPU, and every launch reports that no
// device is present, as the real launchers do on a machine without a GPU.
// Test infrastructure only; never linked into the product library.
#include "../../paper_2606_07713_amd/csrc/launch.h"
#include "../../paper_2606_07713_amd/csrc/proj.h"

namespace moa {

hipError_t launch_prefill_bf16(const Problem&, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_prefill_f32(const Problem&, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_decode(const Problem&, int, float*, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_split_combine(const Problem&, int, const float*, const float*, hipStream_t) {
    return hipErrorNoDevice;
}
hipError_t launch_bwd(const BwdProblem&, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_proj(const ProjProblem&, hipStream_t) { return hipErrorNoDevice; }
hipError_t noalloc_scratch(hipStream_t, void**) { return hipErrorNoDevice; }
hipError_t launch_prefill_gather(const Problem&, const GatherLayout&, hipStream_t) {
    return hipErrorNoDevice;
}

}  // namespace moa
