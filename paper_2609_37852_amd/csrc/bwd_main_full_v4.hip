// Main backward kernel without the mask, protected dP (dP from BF16
// operands): the head-dim pairs whose BF16 tiles fit the LDS (64, 128 and
// 192/128), with and without row statistics.
#include "bwd_main.hpp"

namespace afp8 {
template hipError_t launch_bwd_main<false, 4>(const AttnArgs&, int, int, dim3, hipStream_t);
}  // namespace afp8
