// MFMA-tiled PnP-Nystra kernels (placeholder until the tiled family lands).
#include "internal.hpp"

namespace nystra {

bool tiled_supported(const Problem &) { return false; }

hipError_t launch_tiled_forward(const Problem &, hipStream_t) { return hipErrorInvalidValue; }

}  // namespace nystra
