// Stand-ins for the kernel launchers, so that the host layer (host_api.cpp) can
// be built and run alone, on the CPU, under the address and undefined-behaviour
// sanitizers.  Every launcher reports a failed launch, which the host layer
// must turn into SPARSTAR_ERR_HIP.
#include "../../paper_2608_10519_amd/csrc/launch.h"

namespace sparstar {

hipError_t launch_pool(const PoolArgs&, int, int, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_score(const ScoreArgs&, int, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_select(const SelectArgs&, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_score_select(const ScoreSelectArgs&, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_attn(const AttnArgs&, int, int, bool, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_retained_mass(const float*, const float*, int64_t, float*, hipStream_t) {
  return hipErrorInvalidValue;
}
hipError_t launch_topk_mass(const TopkArgs&, int, hipStream_t) { return hipErrorInvalidValue; }

}  // namespace sparstar
