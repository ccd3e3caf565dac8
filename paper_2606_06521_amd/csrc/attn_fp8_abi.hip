// C ABI of libattn_fp8.so (declared in include/attn_fp8.h): argument
// validation, choice of kernel instantiation, grid sizing, launch on the
// caller's stream.  No per-call state is kept; the only memory taken is the
// prefill kernel's split workspace, one per (device, stream), allocated in
// stream order on first use and kept until the process ends.
#include "../../include/attn_fp8.h"
#include "attn_common.hpp"
#include "attn_launch.hpp"

#include <math.h>
#include <stdint.h>

namespace {

constexpr int kVersion = 510;   // 0.5.1: KV-cache prefill tiles split over workgroups

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

// Shared validation and dispatch of both entry points.
// N: query rows, Nk: cached keys (N for self-attention; N <= Nk, row r at key r + Nk - N)
int run(const void* q, const void* k, const void* v, float* out, float* lse,
        uint32_t* counts, bool count, int B, int Hq, int Hkv, int N, int Nk, int d, int causal,
        int block_kv, int order, float S, int mode_flags, int n_sink, float q_descale,
        float k_descale, float v_descale, void* stream, uint32_t* gap_hist = nullptr,
        uint32_t* blk_zero = nullptr, int nbins = 0)
{
    const int mode = mode_flags & ~ATTN_SCALE_DYNAMIC;
    const bool dyn = (mode_flags & ATTN_SCALE_DYNAMIC) != 0;
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
    if (n_sink < 0)
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
    if (d < 1 || block_kv < 1)
        return ATTN_ERR_INVALID_ARG;
    if (d != 64 && d != 128)
        return ATTN_ERR_UNSUPPORTED;
    if (block_kv != 64 && block_kv != 128)
        return ATTN_ERR_UNSUPPORTED;
    const int64_t rows = (int64_t)B * Hq * N;
    if (rows == 0)
        return ATTN_OK;
    if (!q || !k || !v)
        return ATTN_ERR_INVALID_ARG;
    if (count ? !counts : !out)
        return ATTN_ERR_INVALID_ARG;
    // the kernels move q, k, v and out in 16-byte vectors, lse and counts in
    // 4-byte words (every row of a contiguous tensor then stays aligned)
    auto misaligned = [](const void* ptr, uintptr_t a) { return ptr && ((uintptr_t)ptr % a) != 0; };
    if (misaligned(q, 16) || misaligned(k, 16) || misaligned(v, 16) || misaligned(out, 16) ||
        misaligned(lse, 4) || misaligned(counts, 4) || misaligned(gap_hist, 4) || misaligned(blk_zero, 4))
        return ATTN_ERR_INVALID_ARG;
    if ((gap_hist || blk_zero) && (!count || !gap_hist || !blk_zero || nbins < 1 || nbins > 64))
        return ATTN_ERR_INVALID_ARG;
    // element offsets stay within 64-bit; the grid must fit a 1-D launch
    const bool fast = mode == ATTN_MODE_FAST || mode == ATTN_MODE_FP8QK;
    // Queries against a longer KV cache (fast modes): long query chunks whose
    // offset Nk - N is a multiple of the block run on the persistent kernel
    // (every 32-row wave then still lies in one block of key positions);
    // short ones, or unaligned offsets, on the prefill kernel, whose waves
    // share a 32-row tile's KV blocks.
    const bool prefill = fast && Nk != N && (N < 128 || (Nk - N) % block_kv != 0);
    const int bm = prefill ? attn::prefill_rows_per_wg()
                           : fast ? attn::fast_rows_per_wg(d, block_kv) : attn::faithful_rows_per_wg();
    const int64_t n_tiles = ((int64_t)N + bm - 1) / bm;
    const int64_t total = (int64_t)B * Hq * n_tiles;
    if (total > (int64_t)1 << 30)
        return ATTN_ERR_UNSUPPORTED;

    attn::Params p;
    p.q = q;
    p.k = k;
    p.v = v;
    p.out = out;
    p.lse = lse;
    p.counts = counts;
    p.gap_hist = gap_hist;
    p.blk_zero = blk_zero;
    p.nbins = nbins;
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
    p.ws_max = nullptr;
    p.ws_part = nullptr;

    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e;
    int dev = 0, n_cu = 0;
    if (fast && (hipGetDevice(&dev) != hipSuccess ||
                 hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess))
        return ATTN_ERR_HIP;
    if (gap_hist) {
        const int64_t nz = (int64_t)B * Hq * p.nblk_all;
        hipLaunchKernelGGL(zero_u32, dim3(1024), dim3(256), 0, s, gap_hist, nz * nbins);
        hipLaunchKernelGGL(zero_u32, dim3(1024), dim3(256), 0, s, blk_zero, nz);
        if (hipGetLastError() != hipSuccess)
            return ATTN_ERR_HIP;
    }
    if (prefill) {
        const bool pow2 = is_pow2_scale(S) && S <= 256.0f;
        const int scale = dyn ? attn::kScaleDynamic : pow2 ? attn::kScalePow2 : attn::kScaleAny;
        e = attn::launch_prefill(p, d, block_kv, causal != 0, count, scale,
                                 mode == ATTN_MODE_FP8QK, n_cu, s);
    } else if (fast) {
        // the scaled convert applies 1/S exactly only for S = 2^k, and only
        // below the E4M3 range limit (it does not saturate)
        const bool pow2 = is_pow2_scale(S) && S <= 256.0f;
        const int scale = dyn ? attn::kScaleDynamic : pow2 ? attn::kScalePow2 : attn::kScaleAny;
        // persistent grid: one workgroup per CU (the LDS footprint admits no
        // second one), 8 XCDs, never more workgroups than work units
        const long long per_xcd_max = n_cu >= attn::kNumXcd ? n_cu / attn::kNumXcd : 1;
        const long long per_xcd = p.units / attn::kNumXcd + 1 < per_xcd_max ? p.units / attn::kNumXcd + 1
                                                                            : per_xcd_max;
        const int grid = (int)(per_xcd * attn::kNumXcd);
        e = mode == ATTN_MODE_FP8QK
                ? attn::launch_fast_qk8(p, grid, d, block_kv, causal != 0, count, scale, s)
                : attn::launch_fast(p, grid, d, block_kv, causal != 0, count, scale, s);
    } else {
        e = attn::launch_faithful(p, d, block_kv, causal != 0, count, mode == ATTN_MODE_FAITHFUL, dyn, s);
    }
    return e == hipSuccess ? ATTN_OK : ATTN_ERR_HIP;
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

int attn_fp8_fwd_kv(const void* q, const void* k, const void* v, float* out, float* lse, int B,
                    int Hq, int Hkv, int Nq, int Nk, int d, int causal, int block_kv, int order,
                    float S, int mode, float q_descale, float k_descale, float v_descale,
                    void* stream)
{
    return run(q, k, v, out, lse, nullptr, false, B, Hq, Hkv, Nq, Nk, d, causal, block_kv, order,
               S, mode, 0, q_descale, k_descale, v_descale, stream);
}

int attn_fp8_p_underflow_count_kv(const void* q, const void* k, const void* v, int B, int Hq,
                                  int Hkv, int Nq, int Nk, int d, int causal, int block_kv,
                                  int order, float S, int mode, int n_sink, float q_descale,
                                  float k_descale, float v_descale, uint32_t* counts, float* out,
                                  float* lse, void* stream)
{
    return run(q, k, v, out, lse, counts, true, B, Hq, Hkv, Nq, Nk, d, causal, block_kv, order,
               S, mode, n_sink, q_descale, k_descale, v_descale, stream);
}

const char* attn_fp8_strerror(int status)
{
    switch (status) {
    case ATTN_OK:
        return "ok";
    case ATTN_ERR_INVALID_ARG:
        return "invalid argument (null pointer, bad shape, Hq % Hkv != 0, S not finite "
               "and positive, Nq > Nk, or order/mode/causal/n_sink out of range; the dynamic scale "
               "needs S = 2^k with 0 <= k <= 8; descales must be finite and positive; "
               "the block diagnostic needs all three arrays and 1 <= nbins <= 64; q, k, v and "
               "out must be 16-byte aligned, lse and counts 4-byte aligned)";
    case ATTN_ERR_UNSUPPORTED:
        return "unsupported configuration (d and block_kv must be 64 or 128)";
    case ATTN_ERR_HIP:
        return "the HIP runtime rejected the kernel launch";
    default:
        return "unknown status";
    }
}

int attn_fp8_version(void) { return kVersion; }

}  // extern "C"
