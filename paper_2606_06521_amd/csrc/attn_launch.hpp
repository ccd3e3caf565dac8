// Host-side launchers of the two kernel families (defined next to their
// kernels) and the tile geometry the dispatcher needs to size the grid.
#pragma once

#include "attn_common.hpp"

namespace attn {

hipError_t launch_faithful(const Params& p, int d, int block_kv, bool causal, bool count,
                           bool cast, bool dynamic, hipStream_t stream);
int faithful_rows_per_wg();

// grid: a multiple of 8 workgroups, at most one per CU (persistent kernel)
hipError_t launch_fast(const Params& p, int grid, int d, int block_kv, bool causal, bool count,
                       int scale /* kScale* */, hipStream_t stream);
// the same kernel with E4M3 Q and K (S^T on the FP8 MFMA)
hipError_t launch_fast_qk8(const Params& p, int grid, int d, int block_kv, bool causal, bool count,
                           int scale /* kScale* */, hipStream_t stream);
int fast_rows_per_wg(int d, int block_kv);

// queries against a longer KV cache (p.Nk > p.N), fast modes: one workgroup
// per (batch, head, 32-row query tile), or several per tile when the tiles
// cannot fill n_cu compute units (two launches and a temporary workspace on
// the stream); sets its own grid, nsplit and workspace fields of p
hipError_t launch_prefill(const Params& p, int d, int block_kv, bool causal, bool count, int scale,
                          bool qk8, int n_cu, hipStream_t stream);
int prefill_rows_per_wg();

}  // namespace attn
