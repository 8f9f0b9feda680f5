// Tiled grouped expert GEMMs for prefill shapes (many rows per expert), gfx950.
#include "common.hpp"
#include "launch.hpp"

namespace moe {

bool tiled_supported(int, int) { return false; }

hipError_t launch_tiled_up(const UpArgs&, hipStream_t) { return hipErrorNotSupported; }

hipError_t launch_tiled_down(const DownArgs&, hipStream_t) { return hipErrorNotSupported; }

}  // namespace moe
