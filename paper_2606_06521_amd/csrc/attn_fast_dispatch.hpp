// Launcher of the fast kernel for one (score type, schedule) pair: picks the
// instantiation for (d, block_kv, causal, count, scale).  Each pair is
// instantiated in its own translation unit (attn_fast*.hip) so the heavy
// templates compile in parallel.
#pragma once

#include "attn_fast_kernel.hpp"

namespace attn {

namespace fast_dispatch {

template <int D, int BC, bool CAUSAL, bool COUNT, int SCALE, bool QK8, bool PAIR>
hipError_t launch_one(const Params& p, int grid, hipStream_t stream)
{
    hipLaunchKernelGGL((fast_kernel<D, BC, CAUSAL, COUNT, SCALE, QK8, PAIR>), dim3(grid), dim3(512), 0, stream, p);
    return hipGetLastError();
}

template <int D, int BC, bool CAUSAL, bool COUNT, bool QK8, bool PAIR>
hipError_t launch_scale(const Params& p, int g, int scale, hipStream_t s)
{
    if (scale == kScaleDynamic)
        return launch_one<D, BC, CAUSAL, COUNT, kScaleDynamic, QK8, PAIR>(p, g, s);
    if (scale == kScalePow2)
        return launch_one<D, BC, CAUSAL, COUNT, kScalePow2, QK8, PAIR>(p, g, s);
    return launch_one<D, BC, CAUSAL, COUNT, kScaleAny, QK8, PAIR>(p, g, s);
}

template <int D, int BC, bool QK8, bool PAIR>
hipError_t launch_d_bc(const Params& p, int g, bool causal, bool count, int scale, hipStream_t s)
{
    if (causal)
        return count ? launch_scale<D, BC, true, true, QK8, PAIR>(p, g, scale, s)
                     : launch_scale<D, BC, true, false, QK8, PAIR>(p, g, scale, s);
    return count ? launch_scale<D, BC, false, true, QK8, PAIR>(p, g, scale, s)
                 : launch_scale<D, BC, false, false, QK8, PAIR>(p, g, scale, s);
}

}  // namespace fast_dispatch

template <bool QK8, bool PAIR>
hipError_t launch_fast_t(const Params& p, int grid, int d, int block_kv, bool causal, bool count, int scale,
                         hipStream_t stream)
{
    using namespace fast_dispatch;
    if (d == 64)
        return block_kv == 64 ? launch_d_bc<64, 64, QK8, PAIR>(p, grid, causal, count, scale, stream)
                              : launch_d_bc<64, 128, QK8, PAIR>(p, grid, causal, count, scale, stream);
    return block_kv == 64 ? launch_d_bc<128, 64, QK8, PAIR>(p, grid, causal, count, scale, stream)
                          : launch_d_bc<128, 128, QK8, PAIR>(p, grid, causal, count, scale, stream);
}

}  // namespace attn
