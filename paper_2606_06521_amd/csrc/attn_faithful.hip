// Faithful mode: FP32 Q, K, V; only P is rounded to E4M3 values (Sec. 6.1:
// Q, K, V stay in FP32 so that the P-cast is the only quantisation).
//
// Algorithm 1 per query row, 4 waves x 32 rows per workgroup.  Scores and the
// P.V product run on the FP32 MFMA (v_mfma_f32_32x32x2_f32); exp2 is evaluated
// in FP64 and rounded once to FP32; P*S goes through the hardware E4M3
// convert (round to nearest even) and straight back through the hardware
// decode, so the P.V operand holds the exact E4M3 values.  ATTN_MODE_NOCAST
// (CAST = false) skips the convert.  DYN: the dynamic per-block power-of-two
// scale (the cast of each block uses 2^kj instead of S).
//
// This mode exists for parity and precision studies, not speed: K_j and V_j
// are staged through LDS once per block with no prefetch.
#include "attn_common.hpp"
#include "attn_launch.hpp"

#include <math.h>

namespace attn {

template <int D, int BC, bool CAUSAL, bool COUNT, bool CAST, bool DYN>
__global__ void __launch_bounds__(256) faithful_kernel(Params p)
{
    constexpr int NW = 4;
    constexpr int BM = 32 * NW;
    constexpr int KT = BC / 32;       // 32-key S^T tiles per KV block
    constexpr int DH = D / 2;         // d values per lane half in the QK product
    constexpr int DT = D / 32;        // 32-wide d tiles of O^T
    constexpr int KS = D + 4;         // padded LDS row stride of K (floats)
    extern __shared__ __attribute__((aligned(16))) float smem[];
    float* Ks = smem;                 // [BC][KS]
    float* Vs = smem + BC * KS;       // [BC][D]

    int bh, tile;
    if (!map_tile<CAUSAL>(p, bh, tile))
        return;
    const int N = p.N, Nk = p.Nk, qoff = p.qoff;   // query rows, keys, row r at key r + qoff
    const int b = bh / p.Hq;
    const int hq = bh - b * p.Hq;
    const int hk = hq / (p.Hq / p.Hkv);
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = tid >> 6;
    const int n = lane & 31;          // query row within the wave (also MFMA A row)
    const int h = lane >> 5;          // lane half
    const int row0 = tile * BM;
    const int wrow0 = row0 + 32 * w;
    const int row = wrow0 + n;

    const float* Qg = static_cast<const float*>(p.q) + (size_t)bh * N * D;
    const size_t kvoff = ((size_t)b * p.Hkv + hk) * (size_t)Nk * D;
    const float* Kg = static_cast<const float*>(p.k) + kvoff;
    const float* Vg = static_cast<const float*>(p.v) + kvoff;

    // Q^T fragment: lane (n, h) holds Q[row][h*DH .. h*DH + DH)
    float qf[DH];
    if (row < N) {
        const f32x4* qr = reinterpret_cast<const f32x4*>(Qg + (size_t)row * D + h * DH);
#pragma unroll
        for (int i = 0; i < DH / 4; ++i) {
            const f32x4 t = qr[i];
            qf[4 * i + 0] = t[0];
            qf[4 * i + 1] = t[1];
            qf[4 * i + 2] = t[2];
            qf[4 * i + 3] = t[3];
        }
    } else {
#pragma unroll
        for (int i = 0; i < DH; ++i)
            qf[i] = 0.f;
    }

    const int last_row_wg = min(row0 + BM, N) - 1;
    const int nblk = CAUSAL ? (last_row_wg + qoff) / BC + 1 : (Nk + BC - 1) / BC;
    const bool wave_on = wrow0 < N;
    // blocks of the wave's rows (with qoff = 0 all of them lie in one
    // BC-block of rows; otherwise the last block may hold keys for some rows only)
    const int nblk_w = CAUSAL ? (min(wrow0 + 31, N - 1) + qoff) / BC + 1 : nblk;
    const int a_key = a_row_to_key(n);

    const float c = p.c;
    const float S = p.S;
    float m_run = -INFINITY;
    float mc_run = -INFINITY;
    float ell = 0.f;                  // partial sum of this lane half
    f32x16 o[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int r = 0; r < 16; ++r)
            o[dt][r] = 0.f;
    uint32_t cnt0 = 0, cnt1 = 0, cnt2 = 0;

    for (int it = 0; it < nblk; ++it) {
        const int j = (p.order == 0) ? it : nblk - 1 - it;
        const int t0 = j * BC;
        __syncthreads();
        for (int u = tid; u < BC * D / 4; u += NW * 64) {
            const int key = u / (D / 4);
            const int c4 = u - key * (D / 4);
            f32x4 kv = {0.f, 0.f, 0.f, 0.f};
            f32x4 vv = {0.f, 0.f, 0.f, 0.f};
            if (t0 + key < Nk) {
                kv = *reinterpret_cast<const f32x4*>(Kg + (size_t)(t0 + key) * D + 4 * c4);
                vv = *reinterpret_cast<const f32x4*>(Vg + (size_t)(t0 + key) * D + 4 * c4);
            }
            *reinterpret_cast<f32x4*>(Ks + key * KS + 4 * c4) = kv;
            *reinterpret_cast<f32x4*>(Vs + key * D + 4 * c4) = vv;
        }
        __syncthreads();
        if (!wave_on || j >= nblk_w)
            continue;   // this wave's rows have no valid key in block j

        // ---- S^T = K_j Q^T (raw dot products, FP32 MFMA) ----
        f32x16 s[KT];
#pragma unroll
        for (int kt = 0; kt < KT; ++kt) {
#pragma unroll
            for (int r = 0; r < 16; ++r)
                s[kt][r] = 0.f;
            const float* krow = Ks + (32 * kt + a_key) * KS + h * DH;
#pragma unroll
            for (int i = 0; i < DH; i += 4) {
                const f32x4 a4 = *reinterpret_cast<const f32x4*>(krow + i);
                s[kt] = __builtin_amdgcn_mfma_f32_32x32x2f32(a4[0], qf[i + 0], s[kt], 0, 0, 0);
                s[kt] = __builtin_amdgcn_mfma_f32_32x32x2f32(a4[1], qf[i + 1], s[kt], 0, 0, 0);
                s[kt] = __builtin_amdgcn_mfma_f32_32x32x2f32(a4[2], qf[i + 2], s[kt], 0, 0, 0);
                s[kt] = __builtin_amdgcn_mfma_f32_32x32x2f32(a4[3], qf[i + 3], s[kt], 0, 0, 0);
            }
        }

        // ---- mask: keys past the sequence end, keys after the row (causal) ----
        if ((CAUSAL && t0 + BC - 1 > wrow0 + qoff) || t0 + BC > Nk) {
#pragma unroll
            for (int kt = 0; kt < KT; ++kt)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int key = t0 + 32 * kt + 16 * h + r;
                    if (key >= Nk || (CAUSAL && key > row + qoff))
                        s[kt][r] = -INFINITY;
                }
        }

        // ---- m_new = max(m, max Z); alpha = exp(m - m_new) (base 2) ----
        float mx = -INFINITY;
#pragma unroll
        for (int kt = 0; kt < KT; ++kt)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                mx = fmax_f(mx, s[kt][r]);
        mx = fmax_f(mx, other_half(mx));
        const bool vis = mx > -INFINITY;            // the row has a key in this block
        const float m_new = fmax_f(m_run, mx);
        const float mc_new = m_new * c;
        // before the row's first valid key (possible only with qoff > 0 in
        // reverse order) nothing has accumulated: alpha is irrelevant and P
        // must be 0 (x = -inf), not NaN
        const bool none = mc_new == -INFINITY;
        const float alpha = none ? 1.f : (float)exp2((double)(mc_run - mc_new));
        const float nmc = none ? 0.f : -mc_new;
        if (COUNT && p.gap_hist && vis && h == 0 && row < N)
            record_gap(p, bh, j, mx, c, nmc);
        // Dynamic P-scale: this block's rows cast P * 2^kj, kj = k0 +
        // clamp(floor(-xmax), 0, 126 - k0) with xmax = fma(block max, c, -mc),
        // and the decoded value goes back to S units times 2^(k0 - kj) (exact)
        float Sj = S, back = 1.f;
        if (DYN) {
            const float xmax = __builtin_fmaf(mx, c, nmc);
            const float f = __builtin_fminf(__builtin_fmaxf(__builtin_floorf(-xmax), 0.f), (float)(126 - p.k0));
            const int kj = p.k0 + (int)f;
            Sj = __uint_as_float((uint32_t)(127 + kj) << 23);
            back = __uint_as_float((uint32_t)(127 + p.k0 - kj) << 23);
        }

        // ---- P = exp(Z - m_new); l from pre-cast P; P~ = E4M3(P*S) ----
        float lsum = 0.f;
        uint32_t bz = 0;   // zero codes of this block (valid rows and keys)
        float pt[KT][16];
#pragma unroll
        for (int kt = 0; kt < KT; ++kt) {
#pragma unroll
            for (int r = 0; r < 16; r += 2) {
                const float x0 = __builtin_fmaf(s[kt][r], c, nmc);
                const float x1 = __builtin_fmaf(s[kt][r + 1], c, nmc);
                const float p0 = (float)exp2((double)x0);
                const float p1 = (float)exp2((double)x1);
                lsum += p0;
                lsum += p1;
                float y0 = p0 * Sj;
                float y1 = p1 * Sj;
                if (CAST) {
                    // saturate at the largest finite E4M3 value before the convert
                    y0 = __builtin_fminf(y0, 448.f);
                    y1 = __builtin_fminf(y1, 448.f);
                    const int code = __builtin_amdgcn_cvt_pk_fp8_f32(y0, y1, 0, false);
                    if (COUNT) {
                        const int k0 = t0 + 32 * kt + 16 * h + r;
                        const bool z0 = (code & 0xFF) == 0 && k0 < Nk && (!CAUSAL || k0 <= row + qoff);
                        const bool z1 = (code & 0xFF00) == 0 && k0 + 1 < Nk && (!CAUSAL || k0 + 1 <= row + qoff);
                        if (j > 0) {
                            cnt2 += z0 + z1;
                        } else {
                            if (z0) { if (k0 < p.n_sink) ++cnt0; else ++cnt1; }
                            if (z1) { if (k0 + 1 < p.n_sink) ++cnt0; else ++cnt1; }
                        }
                        if (row < N)
                            bz += z0 + z1;
                    }
                    const auto dec = __builtin_amdgcn_cvt_pk_f32_fp8(code, false);
                    y0 = dec[0];
                    y1 = dec[1];
                }
                if (DYN) {
                    y0 *= back;
                    y1 *= back;
                }
                pt[kt][r] = y0;
                pt[kt][r + 1] = y1;
            }
        }
        ell = alpha * ell + lsum;
        if (COUNT && CAST && p.blk_zero)
            record_block_zeros(p, bh, j, bz);

        // ---- O <- alpha O + P~ V_j  (FP32 MFMA on O^T = V^T P~^T) ----
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                o[dt][r] *= alpha;
#pragma unroll
        for (int kt = 0; kt < KT; ++kt) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const float* vrow = Vs + (32 * kt + 16 * h + r) * D + n;
#pragma unroll
                for (int dt = 0; dt < DT; ++dt)
                    o[dt] = __builtin_amdgcn_mfma_f32_32x32x2f32(vrow[32 * dt], pt[kt][r], o[dt], 0, 0, 0);
            }
        }
        m_run = m_new;
        mc_run = mc_new;
    }

    if (!wave_on)
        return;
    // ---- epilogue: O / (S l) ----
    const float ell_row = ell + other_half(ell);
    if (COUNT) {
        cnt0 += other_half_u32(cnt0);
        cnt1 += other_half_u32(cnt1);
        cnt2 += other_half_u32(cnt2);
    }
    if (row < N) {
        const size_t flat = (size_t)bh * N + row;
        if (p.out) {
            const float denom = S * ell_row;
            float* orow = p.out + flat * D;
#pragma unroll
            for (int dt = 0; dt < DT; ++dt)
#pragma unroll
                for (int r4 = 0; r4 < 4; ++r4) {
                    f32x4 v4;
                    v4[0] = o[dt][4 * r4 + 0] / denom * p.v_descale;
                    v4[1] = o[dt][4 * r4 + 1] / denom * p.v_descale;
                    v4[2] = o[dt][4 * r4 + 2] / denom * p.v_descale;
                    v4[3] = o[dt][4 * r4 + 3] / denom * p.v_descale;
                    *reinterpret_cast<f32x4*>(orow + 32 * dt + 8 * r4 + 4 * h) = v4;
                }
        }
        if (h == 0) {
            if (p.lse)
                p.lse[flat] = (float)(((double)mc_run + log2((double)ell_row)) * 0.6931471805599453094);
            if (COUNT) {
                p.counts[3 * flat + 0] = cnt0;
                p.counts[3 * flat + 1] = cnt1;
                p.counts[3 * flat + 2] = cnt2;
            }
        }
    }
}

template <int D, int BC, bool CAUSAL, bool COUNT, bool CAST, bool DYN>
static hipError_t launch_one(const Params& p, hipStream_t stream)
{
    constexpr size_t lds = sizeof(float) * (size_t)BC * ((D + 4) + D);
    auto kern = faithful_kernel<D, BC, CAUSAL, COUNT, CAST, DYN>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess)
        return e;
    const int grid = p.per_xcd * kNumXcd;
    hipLaunchKernelGGL(kern, dim3(grid), dim3(256), lds, stream, p);
    return hipGetLastError();
}

template <int D, int BC, bool CAUSAL, bool COUNT>
static hipError_t launch_cast(const Params& p, bool cast, bool dyn, hipStream_t s)
{
    if (!cast)
        return launch_one<D, BC, CAUSAL, COUNT, false, false>(p, s);
    return dyn ? launch_one<D, BC, CAUSAL, COUNT, true, true>(p, s)
               : launch_one<D, BC, CAUSAL, COUNT, true, false>(p, s);
}

template <int D, int BC>
static hipError_t launch_d_bc(const Params& p, bool causal, bool count, bool cast, bool dyn, hipStream_t s)
{
    if (causal)
        return count ? launch_cast<D, BC, true, true>(p, cast, dyn, s) : launch_cast<D, BC, true, false>(p, cast, dyn, s);
    return count ? launch_cast<D, BC, false, true>(p, cast, dyn, s) : launch_cast<D, BC, false, false>(p, cast, dyn, s);
}

// Without the cast the dynamic scale is the static one (P * 2^kj * 2^(k0-kj)
// = P * S exactly), so ATTN_MODE_NOCAST ignores it.
hipError_t launch_faithful(const Params& p, int d, int block_kv, bool causal, bool count,
                           bool cast, bool dynamic, hipStream_t stream)
{
    if (d == 64)
        return block_kv == 64 ? launch_d_bc<64, 64>(p, causal, count, cast, dynamic, stream)
                              : launch_d_bc<64, 128>(p, causal, count, cast, dynamic, stream);
    return block_kv == 64 ? launch_d_bc<128, 64>(p, causal, count, cast, dynamic, stream)
                          : launch_d_bc<128, 128>(p, causal, count, cast, dynamic, stream);
}

int faithful_rows_per_wg() { return 128; }

}  // namespace attn
