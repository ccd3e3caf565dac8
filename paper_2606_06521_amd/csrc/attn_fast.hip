// bf16 Q/K instantiations of the fast kernel and their launcher.
#include "attn_fast_kernel.hpp"

namespace attn {

namespace {
constexpr bool QK8_INST = false;
}

template <int D, int BC, bool CAUSAL, bool COUNT, int SCALE>
static hipError_t launch_one(const Params& p, int grid, hipStream_t stream)
{
    hipLaunchKernelGGL((fast_kernel<D, BC, CAUSAL, COUNT, SCALE, QK8_INST>), dim3(grid), dim3(512), 0, stream, p);
    return hipGetLastError();
}

template <int D, int BC, bool CAUSAL, bool COUNT>
static hipError_t launch_scale(const Params& p, int g, int scale, hipStream_t s)
{
    if (scale == kScaleDynamic)
        return launch_one<D, BC, CAUSAL, COUNT, kScaleDynamic>(p, g, s);
    if (scale == kScalePow2)
        return launch_one<D, BC, CAUSAL, COUNT, kScalePow2>(p, g, s);
    return launch_one<D, BC, CAUSAL, COUNT, kScaleAny>(p, g, s);
}

template <int D, int BC>
static hipError_t launch_d_bc(const Params& p, int g, bool causal, bool count, int scale, hipStream_t s)
{
    if (causal)
        return count ? launch_scale<D, BC, true, true>(p, g, scale, s) : launch_scale<D, BC, true, false>(p, g, scale, s);
    return count ? launch_scale<D, BC, false, true>(p, g, scale, s) : launch_scale<D, BC, false, false>(p, g, scale, s);
}

hipError_t launch_fast(const Params& p, int grid, int d, int block_kv, bool causal, bool count,
                       int scale, hipStream_t stream)
{
    if (d == 64)
        return block_kv == 64 ? launch_d_bc<64, 64>(p, grid, causal, count, scale, stream)
                              : launch_d_bc<64, 128>(p, grid, causal, count, scale, stream);
    return block_kv == 64 ? launch_d_bc<128, 64>(p, grid, causal, count, scale, stream)
                          : launch_d_bc<128, 128>(p, grid, causal, count, scale, stream);
}



int fast_rows_per_wg(int, int) { return 256; }

}  // namespace attn
