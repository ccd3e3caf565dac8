// Fast mode: bfloat16 Q and K, OCP E4M3 V; the E4M3 P bytes feed the FP8 MFMA.
//
// Algorithm 1 per query row with the kernel semantics of Sec. 6.1; NW waves of
// 32 query rows per workgroup (BM = 32*NW rows), one KV block of BC keys per
// iteration, in forward or reverse block order:
//   S^T = K_j Q^T        v_mfma_f32_32x32x16_bf16, FP32 accumulate (raw dots)
//   m, alpha, P, l       per-lane scalars (one query row per lane)
//   P8 = E4M3(P * S)     v_cvt_pk_fp8_f32 (round to nearest even); for S = 2^k
//                        the scaled convert v_cvt_scalef32_pk_fp8_f32 applies
//                        the exact power-of-two scale inside the convert
//   O^T += V_j^T P8^T    v_mfma_f32_32x32x64_f8f6f4 (E4M3 x E4M3), FP32 accumulate
//   out = O / (S l)
// K_j / V_j go global -> registers (prefetched one block ahead) -> LDS.  V_j is
// transposed on the way (4x4 byte transposes with v_perm_b32) into a
// d-major layout, because both operands of the FP8 MFMA need the key index
// contiguous per lane.  Both LDS tiles are XOR-swizzled so the MFMA operand
// reads (16 bytes per lane) hit distinct banks.
#include "attn_common.hpp"
#include "attn_launch.hpp"

#include <math.h>

namespace attn {

namespace {

// 16-byte chunk swizzle of a K row (key kappa): the eight keys that lanes
// 0..7 (and 8..15, ...) of a wave read together map to eight different chunks.
__device__ inline int k_swz(int key)
{
    return (key & 3) | (((key >> 4) & 1) << 2);
}

// 16-byte chunk swizzle of a V^T row (d index).
template <int BC>
__device__ inline int v_swz(int d)
{
    if constexpr (BC == 128)
        return (d ^ (d >> 3)) & 7;
    else
        return (d >> 1) & 3;
}

// Transpose a 4 (keys) x 4 (bytes) block: a[i] holds 4 consecutive d-bytes of
// key i; out[e] holds byte e of keys 0..3 (key 0 in the low byte).
__device__ inline void transpose4x4(const uint32_t a0, const uint32_t a1, const uint32_t a2,
                                    const uint32_t a3, uint32_t out[4])
{
    const uint32_t t0 = __builtin_amdgcn_perm(a1, a0, 0x05010400u);
    const uint32_t t1 = __builtin_amdgcn_perm(a1, a0, 0x07030602u);
    const uint32_t t2 = __builtin_amdgcn_perm(a3, a2, 0x05010400u);
    const uint32_t t3 = __builtin_amdgcn_perm(a3, a2, 0x07030602u);
    out[0] = __builtin_amdgcn_perm(t2, t0, 0x05040100u);
    out[1] = __builtin_amdgcn_perm(t2, t0, 0x07060302u);
    out[2] = __builtin_amdgcn_perm(t3, t1, 0x05040100u);
    out[3] = __builtin_amdgcn_perm(t3, t1, 0x07060302u);
}

}  // namespace

template <int D, int BC, bool CAUSAL, bool COUNT, bool POW2, int NW>
__global__ void __launch_bounds__(NW * 64) fast_kernel(Params p)
{
    constexpr int BM = 32 * NW;
    constexpr int NT = NW * 64;
    constexpr int KT = BC / 32;                 // 32-key S^T tiles per block
    constexpr int DK = D / 16;                  // bf16 MFMA k-steps over d
    constexpr int DT = D / 32;                  // 32-wide d tiles of O^T
    constexpr int PVS = BC / 64;                // 64-key FP8 MFMA k-steps
    constexpr int KROW = D * 2;                 // bytes per K row
    constexpr int KCH = D / 8;                  // 16-byte chunks per K row
    constexpr int K_UNITS = BC * KCH;
    constexpr int K_PER_T = (K_UNITS + NT - 1) / NT;
    constexpr int V_UNITS = (BC / 4) * (D / 8); // units of 4 keys x 8 d-bytes
    constexpr int V_PER_T = (V_UNITS + NT - 1) / NT;
    static_assert(KCH >= 8, "K swizzle needs at least 8 chunks per row");

    __shared__ __attribute__((aligned(16))) uint8_t Ks[BC * KROW];
    __shared__ __attribute__((aligned(16))) uint8_t Vt[D * BC];

    int bh, tile;
    if (!map_tile<CAUSAL>(p, bh, tile))
        return;
    const int N = p.N;
    const int b = bh / p.Hq;
    const int hq = bh - b * p.Hq;
    const int hk = hq / (p.Hq / p.Hkv);
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = tid >> 6;
    const int n = lane & 31;
    const int h = lane >> 5;
    const int row0 = tile * BM;
    const int wrow0 = row0 + 32 * w;
    const int row = wrow0 + n;

    const uint8_t* Qg = static_cast<const uint8_t*>(p.q) + (size_t)bh * N * KROW;
    const size_t kvrow0 = ((size_t)b * p.Hkv + hk) * (size_t)N;
    const uint8_t* Kg = static_cast<const uint8_t*>(p.k) + kvrow0 * KROW;
    const uint8_t* Vg = static_cast<const uint8_t*>(p.v) + kvrow0 * D;

    // Q^T fragments (B operand): lane (n, h) holds Q[row][16*kk + 8*h .. +8]
    bf16x8 qf[DK];
    if (row < N) {
        const uint8_t* qr = Qg + (size_t)row * KROW;
#pragma unroll
        for (int kk = 0; kk < DK; ++kk)
            qf[kk] = *reinterpret_cast<const bf16x8*>(qr + (16 * kk + 8 * h) * 2);
    } else {
#pragma unroll
        for (int kk = 0; kk < DK; ++kk)
#pragma unroll
            for (int i = 0; i < 8; ++i)
                qf[kk][i] = (__bf16)0.f;
    }

    const int last_row_wg = min(row0 + BM, N) - 1;
    const int nblk = CAUSAL ? last_row_wg / BC + 1 : (N + BC - 1) / BC;
    const bool wave_on = wrow0 < N;
    const int nblk_w = CAUSAL ? min(wrow0 + 31, N - 1) / BC + 1 : nblk;
    const int a_key = a_row_to_key(n);
    const int a_swz = k_swz(a_key);              // same for every 32-key tile

    // ---- global -> register prefetch of one KV block ----
    i32x4 kreg[K_PER_T];
    uint32_t vreg[V_PER_T][8];                   // 4 keys x (lo, hi) dwords
    auto load_block = [&](int j) {
        const int t0 = j * BC;
#pragma unroll
        for (int i = 0; i < K_PER_T; ++i) {
            const int u = tid + i * NT;
            if (K_UNITS % NT == 0 || u < K_UNITS) {
                const int key = u / KCH;
                const int ch = u - key * KCH;
                if (t0 + key < N)
                    kreg[i] = *reinterpret_cast<const i32x4*>(Kg + (size_t)(t0 + key) * KROW + ch * 16);
                else
                    kreg[i] = i32x4{0, 0, 0, 0};
            }
        }
#pragma unroll
        for (int i = 0; i < V_PER_T; ++i) {
            const int u = tid + i * NT;
            if (V_UNITS % NT == 0 || u < V_UNITS) {
                const int kg = u / (D / 8);
                const int dc = u - kg * (D / 8);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int key = t0 + 4 * kg + e;
                    i32x2 t = {0, 0};
                    if (key < N)
                        t = *reinterpret_cast<const i32x2*>(Vg + (size_t)key * D + dc * 8);
                    vreg[i][2 * e] = (uint32_t)t[0];
                    vreg[i][2 * e + 1] = (uint32_t)t[1];
                }
            }
        }
    };
    auto store_block = [&]() {
#pragma unroll
        for (int i = 0; i < K_PER_T; ++i) {
            const int u = tid + i * NT;
            if (K_UNITS % NT == 0 || u < K_UNITS) {
                const int key = u / KCH;
                const int ch = u - key * KCH;
                *reinterpret_cast<i32x4*>(Ks + key * KROW + ((ch ^ k_swz(key)) << 4)) = kreg[i];
            }
        }
#pragma unroll
        for (int i = 0; i < V_PER_T; ++i) {
            const int u = tid + i * NT;
            if (V_UNITS % NT == 0 || u < V_UNITS) {
                const int kg = u / (D / 8);
                const int dc = u - kg * (D / 8);
                uint32_t tl[4], th[4];
                transpose4x4(vreg[i][0], vreg[i][2], vreg[i][4], vreg[i][6], tl);
                transpose4x4(vreg[i][1], vreg[i][3], vreg[i][5], vreg[i][7], th);
                const int kb = 4 * kg;               // first key (byte) of the unit
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int d = 8 * dc + e;
                    const int off = d * BC + ((((kb >> 4) ^ v_swz<BC>(d))) << 4) + (kb & 15);
                    *reinterpret_cast<uint32_t*>(Vt + off) = e < 4 ? tl[e] : th[e - 4];
                }
            }
        }
    };

    const float c = p.c;
    const float S = p.S;
    const float inv_S = p.inv_S;
    float m_run = -INFINITY;
    float mc_run = -INFINITY;
    float ell = 0.f;
    f32x16 o[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int r = 0; r < 16; ++r)
            o[dt][r] = 0.f;
    uint32_t cnt0 = 0, cnt1 = 0, cnt2 = 0;

    load_block(p.order == 0 ? 0 : nblk - 1);
    for (int it = 0; it < nblk; ++it) {
        const int j = (p.order == 0) ? it : nblk - 1 - it;
        const int t0 = j * BC;
        __syncthreads();                 // previous block fully consumed
        store_block();
        if (it + 1 < nblk)
            load_block(p.order == 0 ? it + 1 : nblk - 2 - it);
        __syncthreads();                 // block j resident in LDS
        if (!wave_on || j >= nblk_w)
            continue;

        // ---- S^T = K_j Q^T ----
        f32x16 s[KT];
#pragma unroll
        for (int kt = 0; kt < KT; ++kt) {
#pragma unroll
            for (int r = 0; r < 16; ++r)
                s[kt][r] = 0.f;
            const uint8_t* krow = Ks + (32 * kt + a_key) * KROW;
#pragma unroll
            for (int kk = 0; kk < DK; ++kk) {
                const int ch = 2 * kk + h;
                const bf16x8 a = *reinterpret_cast<const bf16x8*>(krow + ((ch ^ a_swz) << 4));
                s[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[kk], s[kt], 0, 0, 0);
            }
        }

        // ---- mask: keys past the end of the sequence, keys after the row ----
        if ((CAUSAL && j == nblk_w - 1) || t0 + BC > N) {
#pragma unroll
            for (int kt = 0; kt < KT; ++kt)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int key = t0 + 32 * kt + 16 * h + r;
                    if (key >= N || (CAUSAL && key > row))
                        s[kt][r] = -INFINITY;
                }
        }

        // ---- running max, alpha ----
        float mx = -INFINITY;
#pragma unroll
        for (int kt = 0; kt < KT; ++kt)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                mx = fmax_f(mx, s[kt][r]);
        mx = fmax_f(mx, other_half(mx));
        const float m_new = fmax_f(m_run, mx);
        const float mc_new = m_new * c;
        const float alpha = __builtin_amdgcn_exp2f(mc_run - mc_new);
        const float nmc = -mc_new;

        // ---- P, l (pre-cast), E4M3 cast into the B operand of the P.V MFMA ----
        float lsum = 0.f;
        uint32_t pk[KT][4];
#pragma unroll
        for (int kt = 0; kt < KT; ++kt) {
#pragma unroll
            for (int r4 = 0; r4 < 4; ++r4) {
                float pv[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    pv[i] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[kt][4 * r4 + i], c, nmc));
                    lsum += pv[i];
                }
                uint32_t word;
                if constexpr (POW2) {
                    typedef __attribute__((__vector_size__(2 * sizeof(short)))) short s16x2;
                    s16x2 lo = {0, 0};
                    lo = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(lo, pv[0], pv[1], inv_S, false);
                    lo = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(lo, pv[2], pv[3], inv_S, true);
                    word = __builtin_bit_cast(uint32_t, lo);
                } else {
                    const float y0 = __builtin_fminf(pv[0] * S, 448.f);
                    const float y1 = __builtin_fminf(pv[1] * S, 448.f);
                    const float y2 = __builtin_fminf(pv[2] * S, 448.f);
                    const float y3 = __builtin_fminf(pv[3] * S, 448.f);
                    int wv = __builtin_amdgcn_cvt_pk_fp8_f32(y0, y1, 0, false);
                    wv = __builtin_amdgcn_cvt_pk_fp8_f32(y2, y3, wv, true);
                    word = (uint32_t)wv;
                }
                pk[kt][r4] = word;
                if (COUNT) {
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int key = t0 + 32 * kt + 16 * h + 4 * r4 + i;
                        const bool z = ((word >> (8 * i)) & 0xFFu) == 0 && key < N &&
                                       (!CAUSAL || key <= row);
                        if (z) {
                            if (j > 0) ++cnt2;
                            else if (key < p.n_sink) ++cnt0;
                            else ++cnt1;
                        }
                    }
                }
            }
        }
        ell = alpha * ell + lsum;

        // ---- O <- alpha O + P8 V_j ----
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                o[dt][r] *= alpha;
#pragma unroll
        for (int js = 0; js < PVS; ++js) {
            i32x8 bop;
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
                bop[q4] = (int)pk[2 * js][q4];
                bop[4 + q4] = (int)pk[2 * js + 1][q4];
            }
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) {
                const int d = 32 * dt + n;
                const uint8_t* vrow = Vt + d * BC;
                const int sw = v_swz<BC>(d);
                const i32x4 a0 = *reinterpret_cast<const i32x4*>(vrow + (((4 * js + h) ^ sw) << 4));
                const i32x4 a1 = *reinterpret_cast<const i32x4*>(vrow + (((4 * js + 2 + h) ^ sw) << 4));
                const i32x8 aop = {a0[0], a0[1], a0[2], a0[3], a1[0], a1[1], a1[2], a1[3]};
                o[dt] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(aop, bop, o[dt], 0, 0, 0, 0, 0, 0);
            }
        }
        m_run = m_new;
        mc_run = mc_new;
    }

    if (!wave_on)
        return;
    const float ell_row = ell + other_half(ell);
    if (COUNT) {
        cnt0 += other_half_u32(cnt0);
        cnt1 += other_half_u32(cnt1);
        cnt2 += other_half_u32(cnt2);
    }
    if (row < N) {
        const size_t flat = (size_t)bh * N + row;
        if (p.out) {
            const float inv = 1.0f / (S * ell_row);
            float* orow = p.out + flat * D;
#pragma unroll
            for (int dt = 0; dt < DT; ++dt)
#pragma unroll
                for (int r4 = 0; r4 < 4; ++r4) {
                    f32x4 v4;
                    v4[0] = o[dt][4 * r4 + 0] * inv;
                    v4[1] = o[dt][4 * r4 + 1] * inv;
                    v4[2] = o[dt][4 * r4 + 2] * inv;
                    v4[3] = o[dt][4 * r4 + 3] * inv;
                    *reinterpret_cast<f32x4*>(orow + 32 * dt + 8 * r4 + 4 * h) = v4;
                }
        }
        if (h == 0) {
            if (p.lse)
                p.lse[flat] = (mc_run + log2f(ell_row)) * 0.69314718055994531f;
            if (COUNT) {
                p.counts[3 * flat + 0] = cnt0;
                p.counts[3 * flat + 1] = cnt1;
                p.counts[3 * flat + 2] = cnt2;
            }
        }
    }
}

namespace {
constexpr int kFastWaves = 4;
}

template <int D, int BC, bool CAUSAL, bool COUNT, bool POW2>
static hipError_t launch_one(const Params& p, hipStream_t stream)
{
    const int grid = p.per_xcd * kNumXcd;
    hipLaunchKernelGGL((fast_kernel<D, BC, CAUSAL, COUNT, POW2, kFastWaves>), dim3(grid),
                       dim3(kFastWaves * 64), 0, stream, p);
    return hipGetLastError();
}

template <int D, int BC>
static hipError_t launch_d_bc(const Params& p, bool causal, bool count, bool pow2, hipStream_t s)
{
    if (causal) {
        if (count) return pow2 ? launch_one<D, BC, true, true, true>(p, s) : launch_one<D, BC, true, true, false>(p, s);
        return pow2 ? launch_one<D, BC, true, false, true>(p, s) : launch_one<D, BC, true, false, false>(p, s);
    }
    if (count) return pow2 ? launch_one<D, BC, false, true, true>(p, s) : launch_one<D, BC, false, true, false>(p, s);
    return pow2 ? launch_one<D, BC, false, false, true>(p, s) : launch_one<D, BC, false, false, false>(p, s);
}

hipError_t launch_fast(const Params& p, int d, int block_kv, bool causal, bool count,
                       bool pow2_scale, hipStream_t stream)
{
    if (d == 64)
        return block_kv == 64 ? launch_d_bc<64, 64>(p, causal, count, pow2_scale, stream)
                              : launch_d_bc<64, 128>(p, causal, count, pow2_scale, stream);
    return block_kv == 64 ? launch_d_bc<128, 64>(p, causal, count, pow2_scale, stream)
                          : launch_d_bc<128, 128>(p, causal, count, pow2_scale, stream);
}

int fast_rows_per_wg(int, int) { return 32 * kFastWaves; }

}  // namespace attn
