// Main backward kernel, without the mask, three isolated score channels: every
// head-dim pair, with and without row statistics.
#include "bwd_main.hpp"

namespace afp8 {
template hipError_t launch_bwd_main<false, 8>(const AttnArgs&, int, int, dim3, hipStream_t);
}  // namespace afp8
