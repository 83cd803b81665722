// The fused encoder's unmasked instantiation (every valid position attends to
// every valid position; one 128-position block), in a translation unit of its
// own: the causal kernel's code is then generated exactly as when it is the only
// instantiation.
#include "encoder_fused_device.h"

namespace tav2 {

hipError_t launch_encoder_fused_unmasked(const fz::Args& a, unsigned grid, hipStream_t st) {
  fz::encoder_fused_kernel<true><<<grid, fz::NT, 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace tav2
