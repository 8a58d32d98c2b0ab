// Main backward kernel, causal, compensated dS formation and block-scaled
// backward probability operand: every head-dim pair, with and without row
// statistics.
#include "bwd_main.hpp"

namespace afp8 {
template hipError_t launch_bwd_main<true, 3>(const AttnArgs&, int, int, dim3, hipStream_t);
}  // namespace afp8
