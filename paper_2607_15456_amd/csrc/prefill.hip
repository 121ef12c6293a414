// Causal prefill attention over the paged latent cache (bf16, MFMA).
#include "lla_device.h"
#include "lla_internal.h"

namespace lla {
hipError_t launch_prefill_bf16(const PrefillArgs&, hipStream_t) { return hipErrorNotSupported; }
}  // namespace lla
