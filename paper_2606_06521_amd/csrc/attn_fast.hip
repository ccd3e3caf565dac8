// bf16 Q/K instantiations of the fast kernel, 256-row schedule.
#include "attn_fast_dispatch.hpp"

namespace attn {
template hipError_t launch_fast_t<false, false>(const Params&, int, int, int, bool, bool, int, hipStream_t);
}  // namespace attn
