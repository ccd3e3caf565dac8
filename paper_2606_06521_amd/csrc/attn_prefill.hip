// KV-cache prefill kernel (fast modes): Nq query rows against Nk cached keys,
// query row r at key position Nk - Nq + r (causal rows see keys up to their
// position).  The shape of the paper's Exp. 1 (q_len = 32 against N = 4096)
// and of a prefill kernel working on a KV cache.
//
// A tile of 32 query rows has only 32 rows of work per KV block, so one wave
// would run the whole key sequence alone.  Here the eight waves of a workgroup
// share the tile's KV blocks instead -- wave w takes a contiguous range of
// the visit order -- without changing what Algorithm 1 computes:
//   pass 1: each wave takes the row maxima of its blocks' scores; the
//           running maximum a row has reached when its visit enters wave w's
//           range is the maximum over the ranges of waves 0..w-1;
//   pass 2: each wave runs Algorithm 1 over its range starting from that
//           running maximum, so every block sees exactly the running maximum
//           of the sequential visit: P = exp2(fma(D, c, -mc)) and its E4M3
//           code are those of the one-wave kernel (counts included);
//   merge:  the eight (O, l) partials are brought to the row's final maximum
//           (one exp2 each) and summed.  Only the FP32 rounding of O and l
//           differs from the sequential chain of alpha products.
// The scores are computed twice (once per pass); K is read twice (the
// counters show both reads reaching HBM at the Exp. 1 shape).
//
// When the tiles alone cannot fill the chip, each tile is split over nsplit
// workgroups (the visit order cut into nsplit * 8 contiguous wave ranges) and
// the passes become two launches:
//   PHASE 1: every wave writes the row maxima of its range to the workspace;
//   PHASE 2: every wave starts from the maximum over all earlier ranges (read
//            back from the workspace), runs Algorithm 1 over its range, and
//            brings its (O, l) to the tile's final maximum; each workgroup
//            writes the sum of its eight waves to the workspace;
//   merge:   a third launch (prefill_merge) adds the nsplit partial sums of
//            each tile in a fixed order and writes out and lse.  The launch
//            boundaries order the phases; no workgroup waits on another.
// PHASE 0 is the one-workgroup kernel with both passes fused.
//
// K fragments (the S^T MFMA's A operand) are read straight from HBM, 16
// bytes per lane, in the key order of a_row_to_key.  Each wave copies the V
// block it multiplies straight into its own LDS region (global_load_lds, no
// register staging), in the XOR-swizzled layout read transposed by
// ds_read_b64_tr_b8 (as in the fast kernel).
#include "attn_common.hpp"
#include "attn_launch.hpp"

#include <math.h>
#include <type_traits>

namespace attn {

namespace {

typedef __attribute__((__vector_size__(2 * sizeof(short)))) short s16x2;

__device__ inline i32x2 read_tr8(const uint8_t* p)
{
    return __builtin_amdgcn_ds_read_tr8_b64_v2i32((__attribute__((address_space(3))) i32x2*)(p));
}

// One 16-byte-per-lane direct load: lane i reads HBM bytes [base + voff, +16)
// and writes LDS bytes [dst + 16 i, +16).  Inline assembly, so that its
// completion is awaited only where the kernel says (s_waitcnt vmcnt(0) before
// the LDS stage is read).  M0 carries the LDS base and is used by nothing
// else in this kernel.
__device__ inline void g2lds(const uint8_t* base, uint32_t voff, const uint8_t* dst)
{
    const uint32_t lds = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) uint8_t*)dst;
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2"
                 :
                 : "s"(__builtin_amdgcn_readfirstlane(lds)), "v"(voff), "s"(base)
                 : "memory");
}

constexpr int kPrefillWaves = 8;

}  // namespace

template <int D, int BC, bool CAUSAL, bool COUNT, int SCALE, bool QK8, int PHASE>
__global__ void __launch_bounds__(64 * kPrefillWaves) prefill_kernel(Params p)
{
    constexpr int NW = kPrefillWaves;
    constexpr int KT = BC / 32;                 // 32-key S^T tiles per block
    constexpr int DK = QK8 ? D / 64 : D / 16;   // S^T MFMA k-steps over d
    constexpr int DT = D / 32;                  // 32-wide d tiles of O^T
    constexpr int PVS = BC / 64;                // 64-key FP8 MFMA k-steps
    constexpr int KROW = QK8 ? D : 2 * D;       // bytes per Q / K row
    constexpr int QSTEP = QK8 ? 64 : 32;        // bytes of a row per k-step
    constexpr int VROW = D;                     // bytes per V row
    constexpr int VCPR = VROW / 16;             // 16-byte chunks per V row
    constexpr int V_BYTES = BC * VROW;          // one wave's V stage
    constexpr int V_NI = V_BYTES / 1024;        // 16-byte-per-lane rounds per stage
    constexpr int V_RPI = 1024 / VROW;          // V rows per round
    constexpr int MERGE_BYTES = NW * 32 * D * 4;
    constexpr int LDS_BYTES = NW * V_BYTES > MERGE_BYTES ? NW * V_BYTES : MERGE_BYTES;
    using QFrag = std::conditional_t<QK8, i32x8, bf16x8>;

    __shared__ __attribute__((aligned(1024))) uint8_t lds[LDS_BYTES];
    __shared__ float tab[NW][32];     // pass 1: each wave's row maxima
    __shared__ float lsh[NW][32];     // merge: each wave's l, at the final maximum
    __shared__ uint32_t csh[32][3];   // merge: counts
    __shared__ float rmax[PHASE == 2 ? 8 * NW : 1][32];   // PHASE 2: the maxima of every range

    // workgroup -> (tile unit, part cidx of C); the C workgroups of a unit are
    // consecutive logical indices inside one XCD's contiguous range
    // (per_xcd is a multiple of C), so they share that XCD's L2
    const int C = PHASE == 0 ? 1 : p.nsplit;
    int unit, cidx;
    {
        const int i = blockIdx.x;
        const int slot = i / kNumXcd;
        if (slot >= p.per_xcd)
            return;
        const int L = (i % kNumXcd) * p.per_xcd + slot;
        if (L >= p.total_wg)
            return;
        unit = L / C;
        cidx = L - unit * C;
    }
    const int bh = unit / p.n_tiles;
    const int tile = unit - bh * p.n_tiles;
    const int Nq = p.N, Nk = p.Nk, qoff = p.qoff;
    const int b = bh / p.Hq;
    const int hq = bh - b * p.Hq;
    const int hk = hq / (p.Hq / p.Hkv);
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int n = lane & 31;
    const int h = lane >> 5;
    const int row = 32 * tile + n;              // every wave holds the same 32 rows
    const int pos = row + qoff;                 // the row's key position
    const int rlast = min(32 * tile + 31, Nq - 1);
    // blocks the tile visits, and this wave's contiguous range g of the visit
    // order (C * NW ranges, part cidx holding ranges cidx NW .. cidx NW + NW - 1)
    const int nbt = CAUSAL ? (rlast + qoff) / BC + 1 : (Nk + BC - 1) / BC;
    const int R = C * NW;
    const int g = cidx * NW + w;
    const int it0 = nbt * g / R, it1 = nbt * (g + 1) / R;
    auto jof = [&](int it) __attribute__((always_inline)) { return p.order == 0 ? it : nbt - 1 - it; };

    const uint8_t* Qg = static_cast<const uint8_t*>(p.q) + (size_t)bh * Nq * KROW;
    const size_t kvrow0 = ((size_t)b * p.Hkv + hk) * (size_t)Nk;
    const uint8_t* Kg = static_cast<const uint8_t*>(p.k) + kvrow0 * KROW;
    const uint8_t* Vg = static_cast<const uint8_t*>(p.v) + kvrow0 * VROW;

    if (tid < 32 * 3)
        csh[tid / 3][tid % 3] = 0u;

    // Q^T fragments (B operand), as in the fast kernel
    QFrag qf[DK];
    if (row < Nq) {
        const uint8_t* qr = Qg + (size_t)row * KROW;
#pragma unroll
        for (int kk = 0; kk < DK; ++kk)
            qf[kk] = *reinterpret_cast<const QFrag*>(qr + QSTEP * kk + (QSTEP / 2) * h);
    } else {
#pragma unroll
        for (int kk = 0; kk < DK; ++kk)
            qf[kk] = QFrag{};
    }

    // ---- S^T = K_j Q^T, K fragments from HBM (key 32 kt + a_row_to_key(n)) ----
    // The MFMAs of one 32-key tile wait on a single round of loads: all DK
    // fragments of tile kt are requested together, one tile ahead (WHOLE: all
    // tiles of the block at once, when the registers allow it), so a block
    // costs KT / 2 .. 1 HBM round trips instead of DK.
    const int a_key = a_row_to_key(n);
    f32x16 s[KT];
    auto mfma_qk = [&](const QFrag& a, int kk, const f32x16& acc) __attribute__((always_inline)) {
        if constexpr (QK8)
            return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, qf[kk], acc, 0, 0, 0, 0, 0, 0);
        else
            return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[kk], acc, 0, 0, 0);
    };
    auto load_tile_j = [&](QFrag* dst, int j, int kt) __attribute__((always_inline)) {
        const uint8_t* kr = Kg + (size_t)min(j * BC + 32 * kt + a_key, Nk - 1) * KROW + (QSTEP / 2) * h;
#pragma unroll
        for (int kk = 0; kk < DK; ++kk)
            dst[kk] = *reinterpret_cast<const QFrag*>(kr + QSTEP * kk);
    };
    // PHASE 2 requests the first two K tiles of a wave's first block (and its
    // V block) before it waits for the range maxima, so that round trip
    // overlaps the one for the maxima; qk then starts from those tiles (pre)
    constexpr int NPRE = KT < 2 ? KT : 2;
    auto qk = [&](int j, auto whole, auto pre) __attribute__((always_inline)) {
        constexpr bool HAS_PRE = !std::is_same_v<decltype(pre), std::false_type>;
        auto load_tile = [&](QFrag* dst, int kt) __attribute__((always_inline)) { load_tile_j(dst, j, kt); };
        if constexpr (decltype(whole)::value) {
            QFrag a[KT][DK];
#pragma unroll
            for (int kt = 0; kt < KT; ++kt)
                load_tile(a[kt], kt);
            // every load of the block is requested before the first MFMA waits
            // (the compiler would otherwise issue each load next to its MFMA,
            // one HBM round trip per k-step)
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int kt = 0; kt < KT; ++kt) {
                s[kt] = mfma_qk(a[kt][0], 0, f32x16{});
#pragma unroll
                for (int kk = 1; kk < DK; ++kk)
                    s[kt] = mfma_qk(a[kt][kk], kk, s[kt]);
            }
        } else {
            QFrag a[2][DK];
            if constexpr (HAS_PRE) {
#pragma unroll
                for (int i = 0; i < NPRE; ++i)
#pragma unroll
                    for (int kk = 0; kk < DK; ++kk)
                        a[i][kk] = pre[i][kk];
            } else {
                load_tile(a[0], 0);
            }
#pragma unroll
            for (int kt = 0; kt < KT; ++kt) {
                if (kt + 1 < KT && (!HAS_PRE || kt + 1 >= NPRE))
                    load_tile(a[(kt + 1) & 1], kt + 1);
                __builtin_amdgcn_sched_barrier(0);
                s[kt] = mfma_qk(a[kt & 1][0], 0, f32x16{});
#pragma unroll
                for (int kk = 1; kk < DK; ++kk)
                    s[kt] = mfma_qk(a[kt & 1][kk], kk, s[kt]);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    };
    // keys past the cache end or past the row's position become -inf
    auto mask = [&](int j) __attribute__((always_inline)) {
        const int t0 = j * BC;
        if ((CAUSAL && t0 + BC - 1 > 32 * tile + qoff) || t0 + BC > Nk) {
            const int lim = (CAUSAL ? min(pos, Nk - 1) : Nk - 1) - t0 - 16 * h;
#pragma unroll
            for (int kt = 0; kt < KT; ++kt)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const uint32_t m = (uint32_t)((lim - (32 * kt + r)) >> 31);
                    s[kt][r] = __uint_as_float((__float_as_uint(s[kt][r]) & ~m) | (0xFF800000u & m));
                }
        }
    };
    auto row_max = [&]() __attribute__((always_inline)) {
        float mx = -INFINITY;
#pragma unroll
        for (int kt = 0; kt < KT; ++kt)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                mx = fmax_f(mx, s[kt][r]);
        return halves_max(mx);
    };

    uint8_t* vst = lds + w * V_BYTES;
    auto vswz = [](int r) __attribute__((always_inline)) { return ((r / (256 / VROW)) & (VCPR / 2 - 1)) * 2; };
    // V_j -> this wave's LDS stage, straight from HBM: round i writes LDS bytes
    // [1024 i, +1024); lane l fills row i V_RPI + l / VCPR at physical chunk
    // l % VCPR, which holds logical chunk (l % VCPR) ^ vswz(row).  Issued at
    // the start of the block (PHASE 2's first block: with the range maxima),
    // so it travels with the K loads of the scores; awaited (vmcnt(0)) just
    // before P.V.  Keys past the cache end read row
    // Nk - 1; their P is 0.  Lane offsets count from the block's first row, so
    // they stay below 2^32 for any number of keys.
    // (V_RPI is a multiple of 256 / VROW and VCPR / 2 divides V_RPI / (256 /
    // VROW), so the swizzle of row i V_RPI + l / VCPR does not depend on i: a
    // block inside the cache takes one lane offset and a uniform row step)
    static_assert(V_RPI % (256 / VROW) == 0 && (V_RPI / (256 / VROW)) % (VCPR / 2) == 0,
                  "the V swizzle repeats every round");
    auto issue_v = [&](int j) __attribute__((always_inline)) {
        const int t0 = j * BC;
        const uint32_t v_voff = (uint32_t)((lane / VCPR) * VROW + 16 * ((lane % VCPR) ^ vswz(lane / VCPR)));
        if (t0 + BC <= Nk) {
#pragma unroll
            for (int i = 0; i < V_NI; ++i)
                g2lds(Vg + (size_t)(t0 + i * V_RPI) * VROW, v_voff, vst + 1024 * i);
        } else {
#pragma unroll
            for (int i = 0; i < V_NI; ++i) {
                const int rv = i * V_RPI + lane / VCPR;
                const int lc = (lane % VCPR) ^ vswz(rv);
                g2lds(Vg + (size_t)t0 * VROW, (uint32_t)(min(t0 + rv, Nk - 1) - t0) * VROW + 16 * lc,
                      vst + 1024 * i);
            }
        }
    };

    // ---- pass 1: row maxima over this wave's blocks ----
    float m_start = -INFINITY, m_final = -INFINITY;
    QFrag kpre[NPRE][DK];
    if constexpr (PHASE != 2) {
        float m1 = -INFINITY;
        for (int it = it0; it < it1; ++it) {
            const int j = jof(it);
            qk(j, std::true_type{}, std::false_type{});
            mask(j);
            m1 = fmax_f(m1, row_max());
        }
        if constexpr (PHASE == 1) {
            if (h == 0)
                p.ws_max[((size_t)unit * R + g) * 32 + n] = m1;
            return;
        }
        if (h == 0)
            tab[w][n] = m1;
        __syncthreads();
#pragma unroll
        for (int v = 0; v < NW; ++v) {
            if (v < w)
                m_start = fmax_f(m_start, tab[v][n]);
            m_final = fmax_f(m_final, tab[v][n]);
        }
    } else {
        // the maxima of every range of the tile, from the PHASE 1 launch: the
        // workgroup stages all R x 32 of them (R <= 8 NW) in LDS with one round
        // of loads, then each wave reduces its prefix and the total, eight
        // ranges per round
        const float* mx = p.ws_max + (size_t)unit * R * 32;
        constexpr int PER = 8 * NW * 32 / (64 * NW);
        float t[PER];
#pragma unroll
        for (int q = 0; q < PER; ++q) {
            const int e = tid + 64 * NW * q;
            t[q] = e < R * 32 ? mx[e] : -INFINITY;
        }
        if (it0 < it1) {
            issue_v(jof(it0));
#pragma unroll
            for (int i = 0; i < NPRE; ++i)
                load_tile_j(kpre[i], jof(it0), i);
        }
#pragma unroll
        for (int q = 0; q < PER; ++q)
            rmax[(tid + 64 * NW * q) / 32][(tid + 64 * NW * q) % 32] = t[q];
        __syncthreads();
        for (int cc = 0; cc < C; ++cc) {
            float v[NW];
#pragma unroll
            for (int u = 0; u < NW; ++u)
                v[u] = rmax[cc * NW + u][n];
#pragma unroll
            for (int u = 0; u < NW; ++u) {
                if (cc * NW + u < g)
                    m_start = fmax_f(m_start, v[u]);
                m_final = fmax_f(m_final, v[u]);
            }
        }
    }

    // ---- pass 2: Algorithm 1 over this wave's range, from the running maximum m_start ----
    const float c = p.c;
    const float S = p.S;
    const float inv_S = p.inv_S;
    float m_run = m_start;
    float mc_run = m_start * c;
    float ell = 0.f;
    f32x16 o[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int r = 0; r < 16; ++r)
            o[dt][r] = 0.f;
    uint32_t pk[KT][4] = {};
    int pv_sb = 127;
    uint32_t cnt0 = 0, cnt1 = 0, cnt2 = 0;

    const int j16 = n & 15;
    const uint32_t v_lane = (uint32_t)(((j16 >> 1) + 16 * h) * VROW + (((n >> 4) | vswz(j16 >> 1)) << 4) +
                                       8 * (j16 & 1));

    // one block of the range; PHASE 2's first block has its V and first K
    // tiles requested already
    auto block = [&](int it, auto first) __attribute__((always_inline)) {
        const int j = jof(it);
        const int t0 = j * BC;
        if constexpr (decltype(first)::value) {
            qk(j, std::false_type{}, kpre);
        } else {
            issue_v(j);
            qk(j, std::false_type{}, std::false_type{});
        }
        mask(j);
        const float mx = row_max();
        const bool vis = mx > -INFINITY;            // the row has a key in this block
        const float m_new = fmax_f(m_run, mx);
        const float mc_new = m_new * c;
        // before the row's first valid key nothing has accumulated: alpha is
        // irrelevant and P must be 0 (x = -inf), not NaN
        const bool none = mc_new == -INFINITY;
        const float alpha = none ? 1.f : __builtin_amdgcn_exp2f(mc_run - mc_new);
        const float nmc = none ? 0.f : -mc_new;
        if (COUNT && p.gap_hist && vis && h == 0 && row < Nq)
            record_gap(p, bh, j, mx, c, nmc);
        float cvt_scale = inv_S;
        if constexpr (SCALE == kScaleDynamic) {
            const float xmax = __builtin_fmaf(mx, c, nmc);
            const float f = __builtin_fminf(__builtin_fmaxf(__builtin_floorf(-xmax), 0.f),
                                            (float)(126 - p.k0));
            const int kj = p.k0 + (int)f;
            cvt_scale = __uint_as_float((uint32_t)(127 - kj) << 23);
            pv_sb = 127 + p.k0 - kj;
        }
#pragma unroll
        for (int kt = 0; kt < KT; ++kt)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                s[kt][r] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[kt][r], c, nmc));
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                o[dt][r] *= alpha;
        float lsum = 0.f;
        uint32_t bz = 0;
#pragma unroll
        for (int kt = 0; kt < KT; ++kt) {
#pragma unroll
            for (int r = 0; r < 16; ++r)
                lsum += s[kt][r];
#pragma unroll
            for (int r4 = 0; r4 < 4; ++r4) {
                const float p0 = s[kt][4 * r4 + 0], p1 = s[kt][4 * r4 + 1];
                const float p2 = s[kt][4 * r4 + 2], p3 = s[kt][4 * r4 + 3];
                uint32_t word;
                if constexpr (SCALE != kScaleAny) {
                    s16x2 lo = __builtin_bit_cast(s16x2, pk[kt][r4]);
                    lo = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(lo, p0, p1, cvt_scale, false);
                    lo = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(lo, p2, p3, cvt_scale, true);
                    word = __builtin_bit_cast(uint32_t, lo);
                } else {
                    int wv = __builtin_amdgcn_cvt_pk_fp8_f32(__builtin_fminf(p0 * S, 448.f),
                                                            __builtin_fminf(p1 * S, 448.f),
                                                            (int)pk[kt][r4], false);
                    wv = __builtin_amdgcn_cvt_pk_fp8_f32(__builtin_fminf(p2 * S, 448.f),
                                                        __builtin_fminf(p3 * S, 448.f), wv, true);
                    word = (uint32_t)wv;
                }
                pk[kt][r4] = word;
                if (COUNT) {
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int key = t0 + 32 * kt + 16 * h + 4 * r4 + i;
                        const bool z = ((word >> (8 * i)) & 0xFFu) == 0 && key < Nk &&
                                       (!CAUSAL || key <= pos) && row < Nq;
                        if (z) {
                            if (j > 0) ++cnt2;
                            else if (key < p.n_sink) ++cnt0;
                            else ++cnt1;
                            ++bz;
                        }
                    }
                }
            }
        }
        ell = alpha * ell + lsum;
        if (COUNT && p.blk_zero)
            record_block_zeros(p, bh, j, bz);
        m_run = m_new;
        mc_run = mc_new;

        // O^T += V_j^T P8^T
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
#pragma unroll
        for (int i = 0; i < PVS * DT; ++i) {
            const int js = i / DT, dt = i % DT;
            const uint8_t* va = vst + (v_lane ^ (uint32_t)(dt << 5)) + 64 * js * VROW;
            const i32x2 r0 = read_tr8(va);
            const i32x2 r1 = read_tr8(va + 8 * VROW);
            const i32x2 r2 = read_tr8(va + 32 * VROW);
            const i32x2 r3 = read_tr8(va + 40 * VROW);
            const i32x8 av = {r0[0], r0[1], r1[0], r1[1], r2[0], r2[1], r3[0], r3[1]};
            i32x8 bop;
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
                bop[q4] = (int)pk[2 * js][q4];
                bop[4 + q4] = (int)pk[2 * js + 1][q4];
            }
            if constexpr (SCALE == kScaleDynamic)
                o[dt] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av, bop, o[dt], 0, 0, 0, 127, 0, pv_sb);
            else
                o[dt] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av, bop, o[dt], 0, 0, 0, 0, 0, 0);
        }
    };
    int it = it0;
    if constexpr (PHASE == 2) {
        if (it < it1) {
            block(it, std::true_type{});
            ++it;
        }
    }
    for (; it < it1; ++it)
        block(it, std::false_type{});

    // ---- merge: bring each wave's (O, l) to the row's final maximum and sum ----
    const float mc_final = m_final * c;
    const float beta = mc_run == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mc_run - mc_final);
    const float ell_w = (ell + other_half(ell)) * beta;
    if (COUNT) {
        cnt0 += other_half_u32(cnt0);
        cnt1 += other_half_u32(cnt1);
        cnt2 += other_half_u32(cnt2);
    }
    __syncthreads();                                   // V stages free for the merge buffer
    float* mbuf = reinterpret_cast<float*>(lds) + w * 32 * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) {
            f32x4 v4;
            v4[0] = o[dt][4 * r4 + 0] * beta;
            v4[1] = o[dt][4 * r4 + 1] * beta;
            v4[2] = o[dt][4 * r4 + 2] * beta;
            v4[3] = o[dt][4 * r4 + 3] * beta;
            *reinterpret_cast<f32x4*>(mbuf + n * D + 32 * dt + 8 * r4 + 4 * h) = v4;
        }
    if (h == 0) {
        lsh[w][n] = ell_w;
        if (COUNT) {
            atomicAdd(&csh[n][0], cnt0);
            atomicAdd(&csh[n][1], cnt1);
            atomicAdd(&csh[n][2], cnt2);
        }
    }
    __syncthreads();
    const float* mb = reinterpret_cast<const float*>(lds);
    if constexpr (PHASE == 2) {
        // this workgroup's sum over its waves (at the tile's final maximum)
        constexpr int PART = 32 * D + 32;
        float* part = p.ws_part + ((size_t)unit * C + cidx) * PART;
        for (int e = tid; e < 32 * D / 4; e += 64 * NW) {
            f32x4 acc = *reinterpret_cast<const f32x4*>(mb + 4 * e);
#pragma unroll
            for (int v = 1; v < NW; ++v) {
                const f32x4 t = *reinterpret_cast<const f32x4*>(mb + v * 32 * D + 4 * e);
                acc[0] += t[0];
                acc[1] += t[1];
                acc[2] += t[2];
                acc[3] += t[3];
            }
            *reinterpret_cast<f32x4*>(part + 4 * e) = acc;
        }
        if (tid < 32) {
            float l = 0.f;
#pragma unroll
            for (int v = 0; v < NW; ++v)
                l += lsh[v][tid];
            part[32 * D + tid] = l;
            if (COUNT && 32 * tile + tid < Nq) {
                // the host clears the counts before a split launch
                const size_t flat = (size_t)bh * Nq + 32 * tile + tid;
                atomicAdd(p.counts + 3 * flat + 0, csh[tid][0]);
                atomicAdd(p.counts + 3 * flat + 1, csh[tid][1]);
                atomicAdd(p.counts + 3 * flat + 2, csh[tid][2]);
            }
        }
        return;
    }
    for (int e = tid; e < 32 * D / 4; e += 64 * NW) {
        const int rr = e / (D / 4);
        const int grow = 32 * tile + rr;
        if (grow >= Nq)
            continue;
        float l = 0.f;
#pragma unroll
        for (int v = 0; v < NW; ++v)
            l += lsh[v][rr];
        f32x4 acc = *reinterpret_cast<const f32x4*>(mb + 4 * e);
#pragma unroll
        for (int v = 1; v < NW; ++v) {
            const f32x4 t = *reinterpret_cast<const f32x4*>(mb + v * 32 * D + 4 * e);
            acc[0] += t[0];
            acc[1] += t[1];
            acc[2] += t[2];
            acc[3] += t[3];
        }
        const size_t flat = (size_t)bh * Nq + grow;
        if (p.out) {
            const float inv = p.v_descale / (S * l);
            f32x4 v4;
            v4[0] = acc[0] * inv;
            v4[1] = acc[1] * inv;
            v4[2] = acc[2] * inv;
            v4[3] = acc[3] * inv;
            *reinterpret_cast<f32x4*>(p.out + flat * D + 4 * (e % (D / 4))) = v4;
        }
    }
    if (tid < 32 && 32 * tile + tid < Nq) {
        const size_t flat = (size_t)bh * Nq + 32 * tile + tid;
        float l = 0.f;
#pragma unroll
        for (int v = 0; v < NW; ++v)
            l += lsh[v][tid];
        if (p.lse)   // lane tid of wave 0 holds row tid: m_final is that row's maximum
            p.lse[flat] = (m_final * c + __builtin_log2f(l)) * 0.6931471805599453f;
        if (COUNT) {
            p.counts[3 * flat + 0] = csh[tid][0];
            p.counts[3 * flat + 1] = csh[tid][1];
            p.counts[3 * flat + 2] = csh[tid][2];
        }
    }
}

// Merge of a split tile: workgroup (tile, g) of 128 threads takes rows
// 4 g .. 4 g + 3 of the tile, one 16-byte piece of a row per thread; the
// nsplit partial sums are added in a fixed order and divided by S l.  lse
// comes from the tile's final row maxima (the largest of its range maxima).
template <int D>
__global__ void __launch_bounds__(128) prefill_merge(Params p)
{
    constexpr int PART = 32 * D + 32;
    constexpr int PIECES = D / 4;               // 16-byte pieces per row
    const int unit = blockIdx.x / 8;
    const int rg = blockIdx.x % 8;
    if (unit >= p.total_wg / p.nsplit)
        return;
    const int C = p.nsplit;
    const int bh = unit / p.n_tiles;
    const int tile = unit - bh * p.n_tiles;
    const int Nq = p.N;
    const int t = threadIdx.x;
    if (t >= 4 * PIECES)
        return;
    const int rr = 4 * rg + t / PIECES;           // row in the tile
    const int piece = t % PIECES;
    const int grow = 32 * tile + rr;
    if (grow >= Nq)
        return;
    const float* base = p.ws_part + (size_t)unit * C * PART;
    f32x4 part[8];
    float lp[8];
#pragma unroll
    for (int cc = 0; cc < 8; ++cc) {
        if (cc < C) {
            part[cc] = *reinterpret_cast<const f32x4*>(base + cc * PART + rr * D + 4 * piece);
            lp[cc] = base[cc * PART + 32 * D + rr];
        }
    }
    // the tile's final maximum (for lse): the row's PIECES threads each take
    // up to MPT of the C * NW range maxima, requested with the partial sums,
    // and then the maximum across the group (exact in any order)
    constexpr int NW = kPrefillWaves;
    constexpr int MPT = (8 * NW + PIECES - 1) / PIECES;
    float mloc = -INFINITY;
    if (p.lse) {
        const float* mx = p.ws_max + (size_t)unit * C * NW * 32 + rr;
#pragma unroll
        for (int i = 0; i < MPT; ++i) {
            const int e = piece + PIECES * i;
            if (e < C * NW)
                mloc = fmax_f(mloc, mx[32 * e]);
        }
    }
    f32x4 acc = part[0];
    float l = lp[0];
#pragma unroll
    for (int cc = 1; cc < 8; ++cc) {
        if (cc < C) {
            acc[0] += part[cc][0];
            acc[1] += part[cc][1];
            acc[2] += part[cc][2];
            acc[3] += part[cc][3];
            l += lp[cc];
        }
    }
    const size_t flat = (size_t)bh * Nq + grow;
    if (p.out) {
        const float inv = p.v_descale / (p.S * l);
        f32x4 v4;
        v4[0] = acc[0] * inv;
        v4[1] = acc[1] * inv;
        v4[2] = acc[2] * inv;
        v4[3] = acc[3] * inv;
        *reinterpret_cast<f32x4*>(p.out + flat * D + 4 * piece) = v4;
    }
    // (a row's threads all return above, or none do: the group is whole here)
    if (p.lse) {
#pragma unroll
        for (int off = PIECES / 2; off > 0; off >>= 1)
            mloc = fmax_f(mloc, __shfl_xor(mloc, off, 64));
        if (piece == 0)
            p.lse[flat] = (mloc * p.c + __builtin_log2f(l)) * 0.6931471805599453f;
    }
}

namespace {

// Clears the counts a split launch adds to.
__global__ void prefill_zero(uint32_t* a, int64_t n)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        a[i] = 0u;
}

template <int D, int BC, bool CAUSAL, bool COUNT, int SCALE, int PHASE>
hipError_t launch_one(const Params& p, bool qk8, hipStream_t s)
{
    const int grid = p.per_xcd * kNumXcd;
    if (qk8)
        hipLaunchKernelGGL((prefill_kernel<D, BC, CAUSAL, COUNT, SCALE, true, PHASE>), dim3(grid),
                           dim3(64 * kPrefillWaves), 0, s, p);
    else
        hipLaunchKernelGGL((prefill_kernel<D, BC, CAUSAL, COUNT, SCALE, false, PHASE>), dim3(grid),
                           dim3(64 * kPrefillWaves), 0, s, p);
    return hipGetLastError();
}

// PHASE 1 computes only maxima: one instantiation per shape, whatever the
// scale and diagnostics
template <int D, int BC, bool CAUSAL, bool COUNT>
hipError_t launch_scale(const Params& p, int scale, bool qk8, int phase, hipStream_t s)
{
    if (phase == 1)
        return launch_one<D, BC, CAUSAL, false, kScaleAny, 1>(p, qk8, s);
    if (phase == 2) {
        if (scale == kScaleDynamic)
            return launch_one<D, BC, CAUSAL, COUNT, kScaleDynamic, 2>(p, qk8, s);
        if (scale == kScalePow2)
            return launch_one<D, BC, CAUSAL, COUNT, kScalePow2, 2>(p, qk8, s);
        return launch_one<D, BC, CAUSAL, COUNT, kScaleAny, 2>(p, qk8, s);
    }
    if (scale == kScaleDynamic)
        return launch_one<D, BC, CAUSAL, COUNT, kScaleDynamic, 0>(p, qk8, s);
    if (scale == kScalePow2)
        return launch_one<D, BC, CAUSAL, COUNT, kScalePow2, 0>(p, qk8, s);
    return launch_one<D, BC, CAUSAL, COUNT, kScaleAny, 0>(p, qk8, s);
}

template <int D, int BC>
hipError_t launch_d_bc(const Params& p, bool causal, bool count, int scale, bool qk8, int phase,
                       hipStream_t s)
{
    if (causal)
        return count ? launch_scale<D, BC, true, true>(p, scale, qk8, phase, s)
                     : launch_scale<D, BC, true, false>(p, scale, qk8, phase, s);
    return count ? launch_scale<D, BC, false, true>(p, scale, qk8, phase, s)
                 : launch_scale<D, BC, false, false>(p, scale, qk8, phase, s);
}

hipError_t launch_phase(const Params& p, int d, int block_kv, bool causal, bool count, int scale,
                        bool qk8, int phase, hipStream_t stream)
{
    if (d == 64)
        return block_kv == 64 ? launch_d_bc<64, 64>(p, causal, count, scale, qk8, phase, stream)
                              : launch_d_bc<64, 128>(p, causal, count, scale, qk8, phase, stream);
    return block_kv == 64 ? launch_d_bc<128, 64>(p, causal, count, scale, qk8, phase, stream)
                          : launch_d_bc<128, 128>(p, causal, count, scale, qk8, phase, stream);
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Tiles (32 query rows of one batch and head) that cannot fill the chip are
// split over C workgroups each: C = min(n_cu / tiles, blocks / 8, 8), so that
// every wave range holds at least one KV block.  The split's workspace holds
// the range maxima (tiles * C * 8 * 32 floats) and, from a 256-byte boundary,
// each workgroup's partial sum (tiles * C * (32 d + 32) floats).  Every entry
// a launch reads is written earlier in the same call, so it needs no clearing.
struct Split {
    long long C;
    size_t off_part, bytes;
};

Split plan_split(const Params& p, int d, int block_kv, bool causal, int n_cu)
{
    const long long units = (long long)p.B * p.Hq * p.n_tiles;
    // blocks the last tile visits (no tile visits more)
    const long long nb_max = causal ? ((long long)p.N - 1 + p.qoff) / block_kv + 1
                                    : ((long long)p.Nk + block_kv - 1) / block_kv;
    Split sp{1, 0, 0};
    if (units < n_cu) {
        long long C = n_cu / units;
        if (C > nb_max / kPrefillWaves)
            C = nb_max / kPrefillWaves;
        if (C > 8)
            C = 8;
        sp.C = C < 1 ? 1 : C;
    }
    if (sp.C > 1) {
        const size_t n_max = (size_t)units * sp.C * kPrefillWaves * 32;
        const size_t n_part = (size_t)units * sp.C * (32 * (size_t)d + 32);
        sp.off_part = align256(n_max * sizeof(float));
        sp.bytes = sp.off_part + align256(n_part * sizeof(float));
    }
    return sp;
}

}  // namespace

size_t prefill_workspace_bytes(const Params& p, int d, int block_kv, bool causal, int n_cu)
{
    return plan_split(p, d, block_kv, causal, n_cu).bytes;
}

// The split runs when the caller's workspace holds at least
// prefill_workspace_bytes(); without one (ws == nullptr) the tiles run unsplit
// (same results, fewer workgroups).
hipError_t launch_prefill(const Params& p_in, int d, int block_kv, bool causal, bool count, int scale,
                          bool qk8, int n_cu, void* ws, size_t ws_bytes, hipStream_t stream)
{
    Params p = p_in;
    p.nsplit = 1;
    p.ws_max = nullptr;
    p.ws_part = nullptr;
    const long long units = (long long)p.B * p.Hq * p.n_tiles;
    Split sp = plan_split(p, d, block_kv, causal, n_cu);
    if (sp.C > 1 && (!ws || ws_bytes < sp.bytes))
        sp.C = 1;
    if (sp.C == 1) {
        p.total_wg = (int)units;
        p.per_xcd = (int)((units + kNumXcd - 1) / kNumXcd);
        return launch_phase(p, d, block_kv, causal, count, scale, qk8, 0, stream);
    }
    const long long C = sp.C;
    p.nsplit = (int)C;
    p.total_wg = (int)(units * C);
    p.per_xcd = (int)((units + kNumXcd - 1) / kNumXcd * C);
    p.ws_max = static_cast<float*>(ws);
    p.ws_part = reinterpret_cast<float*>(static_cast<uint8_t*>(ws) + sp.off_part);
    if (count)
        hipLaunchKernelGGL(prefill_zero, dim3(1024), dim3(256), 0, stream, p.counts,
                           (int64_t)p.B * p.Hq * p.N * 3);
    hipError_t e = hipGetLastError();
    if (e == hipSuccess)
        e = launch_phase(p, d, block_kv, causal, count, scale, qk8, 1, stream);
    if (e == hipSuccess)
        e = launch_phase(p, d, block_kv, causal, count, scale, qk8, 2, stream);
    if (e == hipSuccess) {
        if (d == 64)
            hipLaunchKernelGGL(prefill_merge<64>, dim3((unsigned)(units * 8)), dim3(128), 0, stream, p);
        else
            hipLaunchKernelGGL(prefill_merge<128>, dim3((unsigned)(units * 8)), dim3(128), 0, stream, p);
        e = hipGetLastError();
    }
    return e;
}

int prefill_rows_per_wg() { return 32; }

}  // namespace attn
