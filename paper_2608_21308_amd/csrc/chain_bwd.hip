// Backward chain kernel (placeholder until the reverse chain lands).
#include "chain_common.h"

namespace e2ttt {
hipError_t launch_chain_bwd(const ChainConfig&, const ChainArgs&, long, hipStream_t) {
  return hipErrorInvalidValue;
}
}  // namespace e2ttt
