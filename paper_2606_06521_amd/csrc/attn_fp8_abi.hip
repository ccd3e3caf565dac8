// C ABI of libattn_fp8.so (declared in include/attn_fp8.h): argument
// validation, choice of kernel instantiation, grid sizing, launch on the
// caller's stream.  No state is kept and no memory is allocated: the one
// scratch buffer (the KV-cache split's workspace) is the caller's.
#include "../../include/attn_fp8.h"
#include "attn_common.hpp"
#include "attn_launch.hpp"

#include <math.h>
#include <stdint.h>

#include <algorithm>
#include <mutex>

// Scratch of the allocation-free KV-cache entry point (attn_fp8_fwd_kv_noalloc):
// a file-scope device array, one copy per GPU, resident from the library's
// load on that GPU until the process ends.  The KV-cache split needs at most
// CUs * (32 d + 288) * 4 + 512 bytes (4.5 MB on 256 CUs at d = 128).  Host
// code never names the array in a kernel argument or a copy: it uses the
// per-device address from hipGetSymbolAddress (scratch_on_device below).
constexpr size_t kScratchBytes = (size_t)8 << 20;
__device__ __align__(256) uint8_t scratch[kScratchBytes];

namespace {

constexpr int kVersion = 620;   // 0.6.2: 128-row schedule of the fast kernel (ATTN_TILE_*)

// Clears the diagnostic's output arrays on the caller's stream (a kernel, not
// a memset node, so the call stays safe inside a captured graph).
__global__ void zero_u32(uint32_t* a, int64_t n)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        a[i] = 0u;
}

bool is_pow2_scale(float S)
{
    int e = 0;
    const float m = frexpf(S, &e);
    return m == 0.5f;
}

// One validated call: the launch parameters and the choice of kernel.
struct Call {
    attn::Params p;
    int d, block_kv, mode;
    int tile;   // fast kernel rows per tile asked for: 256, 128 or 0 (chosen at launch)
    bool causal, count, dyn, fast, prefill, empty;
};

// Validation of everything but the pointers, and the launch parameters.
// N: query rows, Nk: cached keys (N for self-attention; N <= Nk, row r at key r + Nk - N)
int prepare(Call& cl, bool count, int B, int Hq, int Hkv, int N, int Nk, int d, int causal,
            int block_kv, int order, float S, int mode_flags, int n_sink, float q_descale,
            float k_descale, float v_descale)
{
    const int mode = mode_flags & ~(ATTN_SCALE_DYNAMIC | ATTN_TILE_256 | ATTN_TILE_128);
    const bool dyn = (mode_flags & ATTN_SCALE_DYNAMIC) != 0;
    if ((mode_flags & ATTN_TILE_256) && (mode_flags & ATTN_TILE_128))
        return ATTN_ERR_INVALID_ARG;
    cl.tile = (mode_flags & ATTN_TILE_256) ? 256 : (mode_flags & ATTN_TILE_128) ? 128 : 0;
    if (B < 0 || Hq < 1 || Hkv < 1 || N < 0 || Nk < N || Hq % Hkv != 0)
        return ATTN_ERR_INVALID_ARG;
    if (causal != 0 && causal != 1)
        return ATTN_ERR_INVALID_ARG;
    if (order != ATTN_ORDER_FORWARD && order != ATTN_ORDER_REVERSE)
        return ATTN_ERR_INVALID_ARG;
    if (mode != ATTN_MODE_FAITHFUL && mode != ATTN_MODE_FAST && mode != ATTN_MODE_NOCAST &&
        mode != ATTN_MODE_FP8QK)
        return ATTN_ERR_INVALID_ARG;
    if (!(q_descale > 0.0f) || !isfinite(q_descale) || !(k_descale > 0.0f) || !isfinite(k_descale) ||
        !(v_descale > 0.0f) || !isfinite(v_descale))
        return ATTN_ERR_INVALID_ARG;
    if (!(S > 0.0f) || !isfinite(S))
        return ATTN_ERR_INVALID_ARG;
    if (d < 1 || block_kv < 1)
        return ATTN_ERR_INVALID_ARG;
    // the count categories (sink keys, the rest of the sink's block, the
    // other blocks) are disjoint only while the sink keys fit in block 0
    if (n_sink < 0 || n_sink > block_kv)
        return ATTN_ERR_INVALID_ARG;
    // the dynamic scale keeps S = 2^k0 as its floor, 0 <= k0 <= 8
    int k0 = 0;
    if (dyn) {
        int e = 0;
        const float f = frexpf(S, &e);
        k0 = e - 1;
        if (f != 0.5f || k0 < 0 || k0 > 8)
            return ATTN_ERR_INVALID_ARG;
    }
    if (d != 64 && d != 128)
        return ATTN_ERR_UNSUPPORTED;
    if (block_kv != 64 && block_kv != 128)
        return ATTN_ERR_UNSUPPORTED;
    // key positions plus a block stay inside int
    if (Nk > (1 << 30))
        return ATTN_ERR_UNSUPPORTED;
    const int64_t rows = (int64_t)B * Hq * N;
    cl.empty = rows == 0;
    cl.d = d;
    cl.block_kv = block_kv;
    cl.mode = mode;
    cl.causal = causal != 0;
    cl.count = count;
    cl.dyn = dyn;
    cl.fast = mode == ATTN_MODE_FAST || mode == ATTN_MODE_FP8QK;
    // Queries against a longer KV cache (fast modes): long query chunks whose
    // offset Nk - N is a multiple of the block run on the persistent kernel
    // (every 32-row wave then still lies in one block of key positions);
    // short ones, or unaligned offsets, on the prefill kernel, whose waves
    // share a 32-row tile's KV blocks.
    cl.prefill = cl.fast && Nk != N && (N < 128 || (Nk - N) % block_kv != 0);
    // (the fast kernel's tiles are counted at 256 rows here; a launch that
    // picks the 128-row schedule recounts them)
    const int bm = cl.prefill ? attn::prefill_rows_per_wg()
                              : cl.fast ? attn::kFastRows : attn::faithful_rows_per_wg();
    const int64_t n_tiles = ((int64_t)N + bm - 1) / bm;
    const int64_t total = (int64_t)B * Hq * n_tiles;
    // element offsets stay within 64-bit; the grid must fit a 1-D launch
    if (total > (int64_t)1 << 30)
        return ATTN_ERR_UNSUPPORTED;

    attn::Params& p = cl.p;
    p = attn::Params{};
    p.nblk_all = (int)(((int64_t)Nk + block_kv - 1) / block_kv);
    p.Nk = Nk;
    p.qoff = Nk - N;
    p.B = B;
    p.Hq = Hq;
    p.Hkv = Hkv;
    p.N = N;
    p.order = order;
    p.n_sink = n_sink;
    p.S = S;
    p.inv_S = 1.0f / S;
    p.k0 = k0;
    // exp(z) = exp2(D * c) with z = D qd kd / sqrt(d) (D the raw dot of the
    // stored values, qd and kd the per-tensor descales): c rounded once from double
    p.c = (float)(1.4426950408889634074 * (double)q_descale * (double)k_descale / sqrt((double)d));
    p.v_descale = v_descale;
    p.n_tiles = (int)n_tiles;
    p.total_wg = (int)total;
    p.per_xcd = (int)((total + attn::kNumXcd - 1) / attn::kNumXcd);
    p.pairs = (int)((n_tiles + 1) / 2);
    p.units = (long long)B * Hq * p.pairs;
    p.nsplit = 1;
    return ATTN_OK;
}

int device_cus(int& n_cu)
{
    int dev = 0;
    n_cu = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return ATTN_ERR_HIP;
    return ATTN_OK;
}

// Workspace bytes a prepared call can use (the KV-cache split), on n_cu CUs.
size_t workspace_bytes(const Call& cl, int n_cu)
{
    return cl.prefill ? attn::prefill_workspace_bytes(cl.p, cl.d, cl.block_kv, cl.causal, n_cu) : 0;
}

// Validation of the pointers of a prepared, non-empty call.
int check_pointers(const Call& cl, const void* q, const void* k, const void* v, const float* out,
                   const float* lse, const uint32_t* counts, const uint32_t* gap_hist,
                   const uint32_t* blk_zero, int nbins, const void* ws)
{
    if (!q || !k || !v)
        return ATTN_ERR_INVALID_ARG;
    if (cl.count ? !counts : !out)
        return ATTN_ERR_INVALID_ARG;
    // the kernels move q, k, v and out in 16-byte vectors, lse and counts in
    // 4-byte words (every row of a contiguous tensor then stays aligned)
    auto misaligned = [](const void* ptr, uintptr_t a) { return ptr && ((uintptr_t)ptr % a) != 0; };
    if (misaligned(q, 16) || misaligned(k, 16) || misaligned(v, 16) || misaligned(out, 16) ||
        misaligned(lse, 4) || misaligned(counts, 4) || misaligned(gap_hist, 4) ||
        misaligned(blk_zero, 4) || misaligned(ws, 256))
        return ATTN_ERR_INVALID_ARG;
    if ((gap_hist || blk_zero) && (!cl.count || !gap_hist || !blk_zero || nbins < 1 || nbins > 64))
        return ATTN_ERR_INVALID_ARG;
    return ATTN_OK;
}

// Critical path of the fast kernel's persistent grid on one schedule, in
// ping-pong phases: the largest sum of unit costs any workgroup takes, with
// the kernel's assignment (XCD x owns units [units x / 8, units (x + 1) / 8),
// its workgroups take every per-th of them).  A tile of the 256-row schedule
// costs two phases per visited block (plus one block's worth for the last
// P.V); one of the 128-row schedule one phase per block (plus two), times
// kPairPhase, the measured length of its phases against the 256-row
// schedule's (every phase of the 128-row schedule carries a K/V copy burst).
constexpr double kPairPhase = 1.15;

double fast_critical_path(const attn::Params& p, bool pair, int block_kv, bool causal, int n_cu)
{
    const int rows = pair ? attn::kFastRowsPair : attn::kFastRows;
    const long long T = ((long long)p.N + rows - 1) / rows;
    const long long per_head = pair ? T : (T + 1) / 2;
    const long long units = (long long)p.B * p.Hq * per_head;
    auto tile_cost = [&](long long t) {
        const long long last = std::min((t + 1) * rows, (long long)p.N) - 1;
        const long long nb = causal ? (last + p.qoff) / block_kv + 1 : ((long long)p.Nk + block_kv - 1) / block_kv;
        return pair ? (double)(nb + 2) * kPairPhase : 2.0 * (double)(nb + 1);
    };
    auto unit_cost = [&](long long u) {
        const long long pr = u % per_head;
        if (pair)
            return tile_cost(pr);
        const long long a = T - 1 - pr;
        return a == pr ? tile_cost(pr) : tile_cost(a) + tile_cost(pr);
    };
    const long long per_xcd_max = n_cu >= attn::kNumXcd ? n_cu / attn::kNumXcd : 1;
    const long long per = std::min(units / attn::kNumXcd + 1, per_xcd_max);
    double worst = 0.0;
    for (int x = 0; x < attn::kNumXcd; ++x) {
        const long long b = units * x / attn::kNumXcd, e = units * (x + 1) / attn::kNumXcd;
        for (long long slot = 0; slot < per; ++slot) {
            double sum = 0.0;
            for (long long u = b + slot; u < e; u += per)
                sum += unit_cost(u);
            worst = std::max(worst, sum);
        }
    }
    return worst;
}

// Enqueues a prepared, validated, non-empty call on stream s.
int launch(Call& cl, const void* q, const void* k, const void* v, float* out, float* lse,
           uint32_t* counts, uint32_t* gap_hist, uint32_t* blk_zero, int nbins, void* ws,
           size_t ws_bytes, int n_cu, hipStream_t s)
{
    attn::Params& p = cl.p;
    p.q = q;
    p.k = k;
    p.v = v;
    p.out = out;
    p.lse = lse;
    p.counts = counts;
    p.gap_hist = gap_hist;
    p.blk_zero = blk_zero;
    p.nbins = nbins;
    if (gap_hist) {
        const int64_t nz = (int64_t)p.B * p.Hq * p.nblk_all;
        hipLaunchKernelGGL(zero_u32, dim3(1024), dim3(256), 0, s, gap_hist, nz * nbins);
        hipLaunchKernelGGL(zero_u32, dim3(1024), dim3(256), 0, s, blk_zero, nz);
        if (hipGetLastError() != hipSuccess)
            return ATTN_ERR_HIP;
    }
    const float S = p.S;
    hipError_t e;
    // the scaled convert applies 1/S exactly only for S = 2^k, and only
    // below the E4M3 range limit (it does not saturate)
    const bool pow2 = is_pow2_scale(S) && S <= 256.0f;
    const int scale = cl.dyn ? attn::kScaleDynamic : pow2 ? attn::kScalePow2 : attn::kScaleAny;
    if (cl.prefill) {
        e = attn::launch_prefill(p, cl.d, cl.block_kv, cl.causal, cl.count, scale,
                                 cl.mode == ATTN_MODE_FP8QK, n_cu, ws, ws_bytes, s);
    } else if (cl.fast) {
        // Schedule: 256-row tiles in causal-balanced pairs, unless the caller
        // asked otherwise or their units leave CUs idle and the 128-row
        // schedule (one tile per unit, two waves per 32-row group) has the
        // shorter critical path.
        bool pair = cl.tile == 128;
        if (cl.tile == 0 && p.units < n_cu)
            pair = fast_critical_path(p, true, cl.block_kv, cl.causal, n_cu) <
                   fast_critical_path(p, false, cl.block_kv, cl.causal, n_cu);
        if (pair) {
            const long long n_tiles = ((long long)p.N + attn::kFastRowsPair - 1) / attn::kFastRowsPair;
            const long long total = (long long)p.B * p.Hq * n_tiles;
            p.n_tiles = (int)n_tiles;
            p.total_wg = (int)total;
            p.per_xcd = (int)((total + attn::kNumXcd - 1) / attn::kNumXcd);
            p.pairs = (int)n_tiles;
            p.units = total;
        }
        // persistent grid: one workgroup per CU (the LDS footprint admits no
        // second one), 8 XCDs, never more workgroups than work units
        const long long per_xcd_max = n_cu >= attn::kNumXcd ? n_cu / attn::kNumXcd : 1;
        const long long per_xcd = p.units / attn::kNumXcd + 1 < per_xcd_max ? p.units / attn::kNumXcd + 1
                                                                            : per_xcd_max;
        const int grid = (int)(per_xcd * attn::kNumXcd);
        const bool qk8 = cl.mode == ATTN_MODE_FP8QK;
        auto go = [&](auto fn) { return fn(p, grid, cl.d, cl.block_kv, cl.causal, cl.count, scale, s); };
        e = qk8 ? (pair ? go(attn::launch_fast_t<true, true>) : go(attn::launch_fast_t<true, false>))
                : (pair ? go(attn::launch_fast_t<false, true>) : go(attn::launch_fast_t<false, false>));
    } else {
        e = attn::launch_faithful(p, cl.d, cl.block_kv, cl.causal, cl.count,
                                  cl.mode == ATTN_MODE_FAITHFUL, cl.dyn, s);
    }
    return e == hipSuccess ? ATTN_OK : ATTN_ERR_HIP;
}

// Device address of `scratch` on the current device, taken once per device
// (with that device current) and kept; nullptr if the runtime refuses.
constexpr int kMaxDevices = 64;
std::mutex scratch_mutex;
void* scratch_ptr[kMaxDevices];

void* scratch_on_device()
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
        return nullptr;
    std::lock_guard<std::mutex> lock(scratch_mutex);
    if (!scratch_ptr[dev]) {
        void* ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess) {
            (void)hipGetLastError();
            return nullptr;
        }
        scratch_ptr[dev] = ptr;
    }
    return scratch_ptr[dev];
}

// Shared validation and dispatch of the entry points.  ws: the caller's
// workspace for the KV-cache split (nullptr: no split); a non-null ws must
// hold at least the bytes attn_fp8_kv_workspace_bytes reports.
int run(const void* q, const void* k, const void* v, float* out, float* lse,
        uint32_t* counts, bool count, int B, int Hq, int Hkv, int N, int Nk, int d, int causal,
        int block_kv, int order, float S, int mode_flags, int n_sink, float q_descale,
        float k_descale, float v_descale, void* stream, uint32_t* gap_hist = nullptr,
        uint32_t* blk_zero = nullptr, int nbins = 0, void* ws = nullptr, size_t ws_bytes = 0)
{
    Call cl;
    int st = prepare(cl, count, B, Hq, Hkv, N, Nk, d, causal, block_kv, order, S, mode_flags,
                     n_sink, q_descale, k_descale, v_descale);
    if (st != ATTN_OK || cl.empty)
        return st;
    st = check_pointers(cl, q, k, v, out, lse, counts, gap_hist, blk_zero, nbins, ws);
    if (st != ATTN_OK)
        return st;
    int n_cu = 0;
    if (cl.fast && (st = device_cus(n_cu)) != ATTN_OK)
        return st;
    if (ws && ws_bytes < workspace_bytes(cl, n_cu))
        return ATTN_ERR_INVALID_ARG;
    return launch(cl, q, k, v, out, lse, counts, gap_hist, blk_zero, nbins, ws, ws_bytes, n_cu,
                  static_cast<hipStream_t>(stream));
}

}  // namespace

extern "C" {

int attn_fp8_fwd(const void* q, const void* k, const void* v, float* out, float* lse, int B,
                 int Hq, int Hkv, int N, int d, int causal, int block_kv, int order, float S,
                 int mode, void* stream)
{
    return run(q, k, v, out, lse, nullptr, false, B, Hq, Hkv, N, N, d, causal, block_kv, order, S,
               mode, 0, 1.0f, 1.0f, 1.0f, stream);
}

int attn_fp8_p_underflow_count(const void* q, const void* k, const void* v, int B, int Hq,
                               int Hkv, int N, int d, int causal, int block_kv, int order,
                               float S, int mode, int n_sink, uint32_t* counts, float* out,
                               float* lse, void* stream)
{
    return run(q, k, v, out, lse, counts, true, B, Hq, Hkv, N, N, d, causal, block_kv, order, S,
               mode, n_sink, 1.0f, 1.0f, 1.0f, stream);
}

int attn_fp8_fwd_descaled(const void* q, const void* k, const void* v, float* out, float* lse,
                          int B, int Hq, int Hkv, int N, int d, int causal, int block_kv,
                          int order, float S, int mode, float q_descale, float k_descale,
                          float v_descale, void* stream)
{
    return run(q, k, v, out, lse, nullptr, false, B, Hq, Hkv, N, N, d, causal, block_kv, order, S,
               mode, 0, q_descale, k_descale, v_descale, stream);
}

int attn_fp8_p_underflow_count_descaled(const void* q, const void* k, const void* v, int B,
                                        int Hq, int Hkv, int N, int d, int causal, int block_kv,
                                        int order, float S, int mode, int n_sink,
                                        float q_descale, float k_descale, float v_descale,
                                        uint32_t* counts, float* out, float* lse, void* stream)
{
    return run(q, k, v, out, lse, counts, true, B, Hq, Hkv, N, N, d, causal, block_kv, order, S,
               mode, n_sink, q_descale, k_descale, v_descale, stream);
}

int attn_fp8_block_gap_diag(const void* q, const void* k, const void* v, int B, int Hq, int Hkv,
                            int N, int d, int causal, int block_kv, int order, float S, int mode,
                            int n_sink, float q_descale, float k_descale, float v_descale,
                            int nbins, uint32_t* gap_hist, uint32_t* blk_zero, uint32_t* counts,
                            float* out, float* lse, void* stream)
{
    if (nbins < 1 || nbins > 64)
        return ATTN_ERR_INVALID_ARG;
    if (B > 0 && Hq > 0 && N > 0 && (!gap_hist || !blk_zero))
        return ATTN_ERR_INVALID_ARG;
    return run(q, k, v, out, lse, counts, true, B, Hq, Hkv, N, N, d, causal, block_kv, order, S,
               mode, n_sink, q_descale, k_descale, v_descale, stream, gap_hist, blk_zero, nbins);
}

int attn_fp8_kv_workspace_bytes(int B, int Hq, int Hkv, int Nq, int Nk, int d, int causal,
                                int block_kv, int mode, size_t* bytes)
{
    if (!bytes)
        return ATTN_ERR_INVALID_ARG;
    *bytes = 0;
    Call cl;
    const int st = prepare(cl, false, B, Hq, Hkv, Nq, Nk, d, causal, block_kv, ATTN_ORDER_FORWARD,
                           256.0f, mode, 0, 1.0f, 1.0f, 1.0f);
    if (st != ATTN_OK || cl.empty || !cl.prefill)
        return st;
    int n_cu = 0;
    if (device_cus(n_cu) != ATTN_OK)
        return ATTN_ERR_HIP;
    *bytes = workspace_bytes(cl, n_cu);
    return ATTN_OK;
}

int attn_fp8_fwd_kv(const void* q, const void* k, const void* v, float* out, float* lse, int B,
                    int Hq, int Hkv, int Nq, int Nk, int d, int causal, int block_kv, int order,
                    float S, int mode, float q_descale, float k_descale, float v_descale,
                    void* workspace, size_t workspace_bytes, void* stream)
{
    return run(q, k, v, out, lse, nullptr, false, B, Hq, Hkv, Nq, Nk, d, causal, block_kv, order,
               S, mode, 0, q_descale, k_descale, v_descale, stream, nullptr, nullptr, 0, workspace,
               workspace_bytes);
}

int attn_fp8_fwd_kv_noalloc(const void* q, const void* k, const void* v, float* out, float* lse,
                            int B, int Hq, int Hkv, int Nq, int Nk, int d, int causal,
                            int block_kv, int order, float S, int mode, float q_descale,
                            float k_descale, float v_descale, void* stream)
{
    Call cl;
    int st = prepare(cl, false, B, Hq, Hkv, Nq, Nk, d, causal, block_kv, order, S, mode, 0,
                     q_descale, k_descale, v_descale);
    if (st != ATTN_OK || cl.empty)
        return st;
    st = check_pointers(cl, q, k, v, out, lse, nullptr, nullptr, nullptr, 0, nullptr);
    if (st != ATTN_OK)
        return st;
    int n_cu = 0;
    if (cl.fast && (st = device_cus(n_cu)) != ATTN_OK)
        return st;
    const size_t need = workspace_bytes(cl, n_cu);
    if (need > kScratchBytes)
        return ATTN_ERR_SCRATCH;
    void* ws = nullptr;
    if (need > 0 && !(ws = scratch_on_device()))
        return ATTN_ERR_HIP;
    return launch(cl, q, k, v, out, lse, nullptr, nullptr, nullptr, 0, ws, ws ? kScratchBytes : 0,
                  n_cu, static_cast<hipStream_t>(stream));
}

int attn_fp8_p_underflow_count_kv(const void* q, const void* k, const void* v, int B, int Hq,
                                  int Hkv, int Nq, int Nk, int d, int causal, int block_kv,
                                  int order, float S, int mode, int n_sink, float q_descale,
                                  float k_descale, float v_descale, uint32_t* counts, float* out,
                                  float* lse, void* workspace, size_t workspace_bytes,
                                  void* stream)
{
    return run(q, k, v, out, lse, counts, true, B, Hq, Hkv, Nq, Nk, d, causal, block_kv, order,
               S, mode, n_sink, q_descale, k_descale, v_descale, stream, nullptr, nullptr, 0,
               workspace, workspace_bytes);
}

const char* attn_fp8_strerror(int status)
{
    switch (status) {
    case ATTN_OK:
        return "ok";
    case ATTN_ERR_INVALID_ARG:
        return "invalid argument (null pointer, bad shape, Hq % Hkv != 0, S not finite "
               "and positive, Nq > Nk, or order/mode/causal out of range, n_sink outside "
               "0..block_kv; the dynamic scale "
               "needs S = 2^k with 0 <= k <= 8; descales must be finite and positive; "
               "the block diagnostic needs all three arrays and 1 <= nbins <= 64; q, k, v and "
               "out must be 16-byte aligned, lse and counts 4-byte aligned, a workspace "
               "256-byte aligned and at least attn_fp8_kv_workspace_bytes long)";
    case ATTN_ERR_UNSUPPORTED:
        return "unsupported configuration (d and block_kv must be 64 or 128)";
    case ATTN_ERR_HIP:
        return "the HIP runtime rejected the kernel launch";
    case ATTN_ERR_SCRATCH:
        return "the allocation-free entry point's fixed scratch (8 MiB per GPU) is smaller "
               "than this shape's KV-cache split needs";
    default:
        return "unknown status";
    }
}

int attn_fp8_version(void) { return kVersion; }

}  // extern "C"
