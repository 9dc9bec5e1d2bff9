#include "common.h"
#include "kernels.h"
namespace msparse {
hipError_t launch_attn_bwd(const AttnArgs&, hipStream_t) { return hipErrorNotSupported; }
}  // namespace msparse
