// E4M3 Q/K instantiations of the fast kernel (S^T on the FP8 MFMA), 256-row
// schedule.
#include "attn_fast_dispatch.hpp"

namespace attn {
template hipError_t launch_fast_t<true, false>(const Params&, int, int, int, bool, bool, int, hipStream_t);
}  // namespace attn
