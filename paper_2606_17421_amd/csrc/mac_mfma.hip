// int8 matrix-core modular MAC (digit-split); kernel not yet enabled.
#include "ckks_internal.hpp"

namespace ckks {

size_t mac_mfma_workspace_bytes(uint32_t, uint32_t, uint32_t) { return 0; }

hipError_t launch_mac_scalar_mfma(const Tables&, const uint32_t*, const uint32_t*, uint32_t*, uint32_t,
                                  uint32_t, uint32_t, void*, hipStream_t) {
  return hipErrorNotSupported;
}

}  // namespace ckks
