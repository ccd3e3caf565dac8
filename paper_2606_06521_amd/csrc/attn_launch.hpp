// Host-side launchers of the two kernel families (defined next to their
// kernels) and the tile geometry the dispatcher needs to size the grid.
#pragma once

#include "attn_common.hpp"

namespace attn {

hipError_t launch_faithful(const Params& p, int d, int block_kv, bool causal, bool count,
                           bool cast, bool dynamic, hipStream_t stream);
int faithful_rows_per_wg();

// The fast kernel (persistent): QK8 selects E4M3 Q and K (S^T on the FP8
// MFMA), PAIR the 128-row schedule (two waves per 32-row group, alternate
// blocks).  grid: a multiple of 8 workgroups, at most one per CU; scale: kScale*.
// Each (QK8, PAIR) pair is instantiated in its own translation unit.
template <bool QK8, bool PAIR>
hipError_t launch_fast_t(const Params& p, int grid, int d, int block_kv, bool causal, bool count, int scale,
                         hipStream_t stream);
extern template hipError_t launch_fast_t<false, false>(const Params&, int, int, int, bool, bool, int, hipStream_t);
extern template hipError_t launch_fast_t<false, true>(const Params&, int, int, int, bool, bool, int, hipStream_t);
extern template hipError_t launch_fast_t<true, false>(const Params&, int, int, int, bool, bool, int, hipStream_t);
extern template hipError_t launch_fast_t<true, true>(const Params&, int, int, int, bool, bool, int, hipStream_t);
// query rows per tile (one work unit of the 128-row schedule, half of one
// of the 256-row schedule's tile pairs)
constexpr int kFastRows = 256;
constexpr int kFastRowsPair = 128;

// queries against a longer KV cache (p.Nk > p.N), fast modes: one workgroup
// per (batch, head, 32-row query tile), or several per tile when the tiles
// cannot fill n_cu compute units and the caller brings a workspace of at least
// prefill_workspace_bytes() (three launches on the stream); sets its own grid,
// nsplit and workspace fields of p
hipError_t launch_prefill(const Params& p, int d, int block_kv, bool causal, bool count, int scale,
                          bool qk8, int n_cu, void* ws, size_t ws_bytes, hipStream_t stream);
// device workspace the split of launch_prefill needs (0: the tiles run unsplit)
size_t prefill_workspace_bytes(const Params& p, int d, int block_kv, bool causal, int n_cu);
int prefill_rows_per_wg();

}  // namespace attn
