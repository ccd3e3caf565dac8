// Shared device-side pieces of the FP8 attention kernels for gfx950 (CDNA4):
// MFMA operand types, the launch parameter block, the XCD-aware mapping of
// workgroups to (batch*head, query tile), and wave-level helpers.
//
// Layout convention used by both kernel families ("transposed" form):
//   S^T = K . Q^T   and   O^T = V^T . P^T
// A 32x32 MFMA accumulator gives lane (n = lane % 32, h = lane / 32) the
// elements D[8*(r/4) + 4*h + (r%4)][n], r = 0..15.  With the query row as the
// N index, every accumulator register of a lane belongs to ONE query row, so
// the running max, the sum l and the rescale factor alpha are per-lane scalars
// and a row reduction needs one exchange between the two 32-lane halves.
// Key rows of the S^T tile are permuted so that register r of half h holds key
// 16*h + r of the 32-key tile; the P bytes of a lane then form the B operand
// of the FP8 P.V MFMA without any data movement.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace attn {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(8 * sizeof(int)))) int i32x8;
typedef __attribute__((__vector_size__(4 * sizeof(int)))) int i32x4;
typedef __attribute__((__vector_size__(2 * sizeof(int)))) int i32x2;

// Launch parameters (passed by value as the kernel argument block).
struct Params {
    const void* q;
    const void* k;
    const void* v;
    float* out;
    float* lse;          // nullable
    uint32_t* counts;    // COUNT instantiations only
    // per-block diagnostic (COUNT instantiations, both nullable):
    // gap_hist[(bh * nblk_all + j) * nbins + bin] counts the rows whose gap
    // g = -fma(block max, c, -mc) (log2 units) has min(max(floor(g), 0),
    // nbins - 1) == bin; blk_zero[bh * nblk_all + j] counts block j's zero codes
    uint32_t* gap_hist;
    uint32_t* blk_zero;
    int nbins;
    int nblk_all;        // ceil(N / block_kv)
    int B, Hq, Hkv, N;   // N: query rows per (batch, head)
    int Nk;              // cached keys per (batch, kv head); N for self-attention
    int qoff;            // Nk - N: query row r sits at key position r + qoff
    int order;           // 0 forward, 1 reverse
    int n_sink;
    float S;             // static P-scale (2^k0 with the dynamic scale)
    float inv_S;         // 1/S, used only when S is a power of two (exact)
    int k0;              // log2 S (dynamic scale only)
    float v_descale;     // per-tensor V descale, applied in the epilogue
    float c;             // fl32(log2(e) / sqrt(d))
    int n_tiles;         // query tiles per (batch, head)
    int total_wg;        // B * Hq * n_tiles
    int per_xcd;         // ceil(total_wg / 8)
    // persistent schedule (fast kernel): a work unit is a pair of query
    // tiles (t, n_tiles - 1 - t) of one (batch, head)
    int pairs;           // units per (batch, head) = ceil(n_tiles / 2)
    long long units;     // B * Hq * pairs
    // prefill kernel split over several workgroups per 32-row tile (nsplit
    // > 1); the workspace is owned by the launcher for the duration of a call
    int nsplit;          // workgroups per tile (1: one fused workgroup)
    float* ws_max;       // [tile][nsplit * waves][32] row maxima of each wave range
    float* ws_part;      // [tile][nsplit][32 * d + 32] each workgroup's O sum, then l
};

// how the fast kernel applies the P-scale
constexpr int kScaleAny = 0;       // static S: multiply, clamp at 448, convert
constexpr int kScalePow2 = 1;      // static S = 2^k <= 256: the scaled convert
constexpr int kScaleDynamic = 2;   // per-block 2^kj (S = 2^k0 its floor)

constexpr int kNumXcd = 8;   // MI355X: 8 XCDs x 32 CUs, workgroup i runs on XCD i % 8

// Workgroup -> (batch*head, tile).  Hardware places workgroup i on XCD i % 8;
// the logical index gives each XCD a contiguous range, so all query tiles of
// one head (and neighbouring heads of one GQA group) run on the same XCD and
// share its L2 for the K/V stream.  Under causal masking the heaviest tile of a
// head (the last rows) is issued first.
template <bool CAUSAL>
__device__ inline bool map_tile(const Params& p, int& bh, int& tile)
{
    const int i = blockIdx.x;
    const int xcd = i % kNumXcd;
    const int slot = i / kNumXcd;
    if (slot >= p.per_xcd)
        return false;
    const int L = xcd * p.per_xcd + slot;
    if (L >= p.total_wg)
        return false;
    bh = L / p.n_tiles;
    const int t = L - bh * p.n_tiles;
    tile = CAUSAL ? (p.n_tiles - 1 - t) : t;
    return true;
}

// Persistent schedule of the fast kernel.  The grid holds one workgroup per
// CU (8 XCDs x gridDim.x / 8 CUs).  Work units -- pairs of query tiles
// (t, T - 1 - t) of one (batch, head) -- are numbered head-major and split
// into 8 contiguous ranges, one per XCD, so the heads of an XCD (and the
// query heads of a GQA group) stream their K/V through one L2.  Inside its
// range a workgroup takes every (gridDim.x / 8)-th unit.  Under causal
// masking a tile pair costs the same for every t (the blocks of tile t plus
// those of tile T - 1 - t), so every CU gets the same amount of work; the
// heavier tile of a pair runs first.
struct UnitRange {
    long long begin, end;   // this XCD's units
    int first, stride;      // first unit offset and stride of this workgroup
};

__device__ inline UnitRange unit_range(const Params& p)
{
    const int xcd = blockIdx.x % kNumXcd;
    const int per = gridDim.x / kNumXcd;
    UnitRange r;
    r.begin = p.units * xcd / kNumXcd;
    r.end = p.units * (xcd + 1) / kNumXcd;
    r.first = blockIdx.x / kNumXcd;
    r.stride = per;
    return r;
}

// Key permutation inside a 32-key S^T tile: MFMA A-row m -> key offset, so that
// accumulator register r of lane half h holds key 16*h + r.
// m = (b4 b3 b2 b1 b0) -> key = (b2 b4 b3 b1 b0).
__device__ inline int a_row_to_key(int m)
{
    return ((m >> 2) & 1) * 16 + ((m >> 3) & 3) * 4 + (m & 3);
}

// Value of the other 32-lane half of the wave.
__device__ inline float other_half(float x)
{
    return __shfl_xor(x, 32, 64);
}

__device__ inline uint32_t other_half_u32(uint32_t x)
{
    return (uint32_t)__shfl_xor((int)x, 32, 64);
}

// Per-block diagnostic of one row: bin of the gap between the running maximum
// and block j's largest score, g = -fma(block max, c, -mc) in log2 units (the
// block's largest P is 2^-g), clamped to [0, nbins - 1]; one count per row.
__device__ inline void record_gap(const Params& p, int bh, int j, float mx, float c, float nmc)
{
    const float g = __builtin_fmaxf(__builtin_floorf(-__builtin_fmaf(mx, c, nmc)), 0.f);
    const int bin = (int)__builtin_fminf(g, (float)(p.nbins - 1));
    atomicAdd(p.gap_hist + ((size_t)bh * p.nblk_all + j) * p.nbins + bin, 1u);
}

// Per-block diagnostic of one wave: adds the wave's zero codes of block j.
__device__ inline void record_block_zeros(const Params& p, int bh, int j, uint32_t z)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1)
        z += (uint32_t)__shfl_xor((int)z, off, 64);
    if ((threadIdx.x & 63) == 0 && z != 0)
        atomicAdd(p.blk_zero + (size_t)bh * p.nblk_all + j, z);
}

// max / sum of a value over the two 32-lane halves (lane i and lane i ^ 32),
// returned in every lane.  v_permlane32_swap with both operands x yields the
// lower-half values and the upper-half values, each in all 64 lanes; the
// symmetric combine does not depend on which result holds which half.
__device__ inline float halves_max(float x)
{
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __builtin_fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ inline float halves_sum(float x)
{
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ inline float fmax_f(float a, float b) { return __builtin_fmaxf(a, b); }

// Number of zero bytes in a word of four E4M3 codes of non-negative values
// (every byte <= 0x7F): adding 0x7F to the low seven bits of a byte sets its
// top bit unless the byte is zero, with no carry into the next byte.
__device__ inline uint32_t zero_codes(uint32_t w)
{
    const uint32_t nz = ((w & 0x7F7F7F7Fu) + 0x7F7F7F7Fu) | w;
    return (uint32_t)__builtin_popcount(~nz & 0x80808080u);
}

}  // namespace attn
