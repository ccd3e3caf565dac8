// The fast kernel (template): bfloat16 Q and K (QK8 = false) or OCP E4M3 Q
// and K (QK8 = true), OCP E4M3 V; the E4M3 P bytes feed the FP8 MFMA.
// Instantiated through attn_fast_dispatch.hpp by attn_fast.hip and
// attn_fast_qk8.hip (256-row tiles) and attn_fast_pair.hip and
// attn_fast_qk8_pair.hip (128-row tiles, PAIR), bf16 and E4M3 Q/K.
//
// Algorithm 1 per query row with the kernel semantics of Sec. 6.1, one KV block
// of BC keys per iteration, in forward or reverse block order:
//   S^T = K_j Q^T        v_mfma_f32_32x32x16_bf16 (bf16) or
//                        v_mfma_f32_32x32x64_f8f6f4 (E4M3, the FP8 x FP8
//                        scores of Algorithm 1), FP32 accumulate (raw dots)
//   m, alpha, P, l       per-lane scalars (one query row per lane)
//   P8 = E4M3(P * S)     v_cvt_pk_fp8_f32 (round to nearest even); for S = 2^k
//                        the scaled convert v_cvt_scalef32_pk_fp8_f32 applies
//                        the exact power-of-two scale inside the convert; the
//                        dynamic per-block scale 2^kj rides on the same convert
//                        (per-lane scale) and on the P.V MFMA's E8M0 B scale
//   O^T += V_j^T P8^T    v_mfma_f32_32x32x64_f8f6f4 (E4M3 x E4M3), FP32 accumulate
//   out = O / (S l)
//
// Schedule ("ping-pong"): 8 waves of 32 query rows; waves w and w+4 share a
// SIMD.  Group 0 (waves 0-3) and group 1 (waves 4-7) alternate between an MFMA
// phase (P.V of the previous block, then S^T of the current block) and a VALU
// phase (max, exp2, l, cast, rescale of O), one phase apart, with a workgroup
// barrier between phases.  On every SIMD one wave keeps the matrix core busy
// while the other runs the softmax.
//
// Grid: persistent, one workgroup per CU; each takes tile pairs (t, T-1-t)
// of the heads of its XCD (unit_range), which equalises the causal work per
// CU.
//
// K_j and V_j go global -> LDS with no register staging
// (global_load_lds_dwordx4, lane i -> LDS base + 16 i), double-buffered, issued
// by group 0 at the start of its MFMA phase two phases before first use.
// K rows are stored in the order the S^T MFMA reads them (a key permutation
// inside each 32-key tile, see a_row_to_key); V stays key-major and is read
// transposed by ds_read_b64_tr_b8, which hands each lane 8 consecutive keys of
// its d column.  Rows are unpadded; the 16-byte chunks of a row are permuted by
// an XOR with a function of the row (kswz / vswz) so that the 16-byte K reads
// and the transposed V reads of a lane group fall in distinct banks.  With
// that layout a loading lane's HBM offset is a per-lane constant plus a
// per-block scalar, so issuing a load costs no vector instructions.
//
// Output (256-row tiles, d = 128): the tile's O goes through the idle K/V
// stages, so each store writes whole 128-byte row segments instead of the
// accumulator layout's 32 rows x 32 bytes.
#pragma once

#include "attn_common.hpp"
#include "attn_launch.hpp"

#include <math.h>
#include <type_traits>

namespace attn {

namespace {

typedef __attribute__((__vector_size__(2 * sizeof(short)))) short s16x2;

// One 16-byte-per-lane direct load: lane i reads HBM bytes [base + voff, +16)
// (base uniform, voff per lane) and writes LDS bytes [dst + 16 i, +16).
// Issued as inline assembly so the compiler does not tie its completion to
// the next barrier; the kernel waits for it explicitly (wait_loads) before
// the barrier that publishes the stage.  M0 holds the wave's LDS base and is
// used by nothing else in this kernel.
__device__ inline void g2lds16(const uint8_t* base, uint32_t voff, uint32_t lds)
{
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2"
                 :
                 : "s"(__builtin_amdgcn_readfirstlane(lds)), "v"(voff), "s"(base)
                 : "memory");
}

// LDS byte address of a pointer into a __shared__ array, or of an LDS address
// already in hand (the 128-row schedule computes its stage addresses so)
__device__ inline uint32_t lds_addr(const uint8_t* p)
{
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) uint8_t*)p;
}
__device__ inline uint32_t lds_addr(uint32_t a) { return a; }

__device__ inline void g2lds16(const uint8_t* base, uint32_t voff, const uint8_t* dst_wave_base)
{
    g2lds16(base, voff, lds_addr(dst_wave_base));
}

__device__ inline void wait_loads()
{
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// LDS load from an integer LDS address
template <typename T>
__device__ inline T lds_load(uint32_t a)
{
    return *reinterpret_cast<const __attribute__((address_space(3))) T*>((uintptr_t)a);
}

// Materialises a per-lane LDS address in one register: the loads that share
// it then carry their constant offsets in the instruction (the 128-row
// schedule's stages move from block to block, so the compiler would otherwise
// keep a register per address and add the stage to each).  Applied to a lane
// offset it also keeps the compiler from hoisting the offset's XOR variants
// out of the loop into registers of their own.
__device__ inline uint32_t lds_base(uint32_t a)
{
    asm volatile("" : "+v"(a));
    return a;
}

__device__ inline i32x2 lds_read_tr8(const uint8_t* p)
{
    return __builtin_amdgcn_ds_read_tr8_b64_v2i32((__attribute__((address_space(3))) i32x2*)(p));
}

}  // namespace

// SCALE: kScaleAny (static S, multiply and convert), kScalePow2 (static
// S = 2^k, the scaled convert) or kScaleDynamic (per-block 2^kj, see softmax).
// PAIR: the 128-row schedule.  Waves w and w + 4 (one per group, on one SIMD)
// share a 32-row group and take alternate blocks of the visit: group g the
// blocks at visit positions k = g, g + 2, ...  The running maximum after
// each block is handed to the partner through LDS, so every block still sees
// the running maximum of the sequential visit (P, its E4M3 code and the counts
// are those of the 256-row schedule); each wave keeps its own (O, l), brought
// to the row's final maximum and added at the end of the tile.  Each tile is
// one work unit (no pairing), which fills the chip when 256-row tiles leave
// CUs idle.
template <int D, int BC, bool CAUSAL, bool COUNT, int SCALE, bool QK8, bool PAIR>
__global__ void __launch_bounds__(512) fast_kernel(Params p)
{
    constexpr int NW = 8;
    constexpr int BM = PAIR ? 32 * (NW / 2) : 32 * NW;
    constexpr int KT = BC / 32;                 // 32-key S^T tiles per block
    constexpr int DK = QK8 ? D / 64 : D / 16;   // S^T MFMA k-steps over d
    constexpr int DT = D / 32;                  // 32-wide d tiles of O^T
    constexpr int PVS = BC / 64;                // 64-key FP8 MFMA k-steps
    constexpr int KROW = QK8 ? D : D * 2;       // bytes per Q / K row (HBM and LDS)
    constexpr int VROW = D;                     // bytes per V row
    constexpr int KCPR = KROW / 16;             // 16-byte chunks per row
    constexpr int VCPR = VROW / 16;
    constexpr int K_BYTES = BC * KROW;          // one K stage
    constexpr int V_BYTES = BC * VROW;
    constexpr int K_RPI = 1024 / KROW;          // rows written by one wave load instruction
    constexpr int V_RPI = 1024 / VROW;
    constexpr int K_NI = K_BYTES / 4096;        // load instructions per loading wave (4 waves)
    constexpr int V_NI = V_BYTES / 4096;
    static_assert(K_NI >= 1 && V_NI >= 1, "stage smaller than one round of loads");

    // 256-row schedule: K stages 0 and 1, then V stages 0 and 1, contiguous
    // (the output tile is staged in [K_BYTES, K_BYTES + 32 KB) at the end)
    __shared__ __attribute__((aligned(1024))) uint8_t Sst[PAIR ? 1 : 2 * (K_BYTES + V_BYTES)];
    // PAIR: two K and two V stages (stage r at Kst + r K_BYTES, Vst +
    // r V_BYTES), and the running maximum of each row (row group w & 3, row n)
    // after the last block processed
    __shared__ __attribute__((aligned(1024))) uint8_t Kst[PAIR ? 2 * K_BYTES : 1];
    __shared__ __attribute__((aligned(1024))) uint8_t Vst[PAIR ? 2 * V_BYTES : 1];
    __shared__ float mslot[PAIR ? NW / 2 : 1][32];

    // Chunk swizzles: LDS row r of a stage stores logical 16-byte chunk L at
    // physical chunk L ^ swz(r).  kswz spreads the 16 rows read by a 16-lane
    // group (one logical chunk) over the 16 bank slots of 256 bytes; vswz does
    // the same for the 8 rows x 2 chunks read by a 32-lane transposed read.
    // Both depend only on row bits below 5, so they are the same for every
    // 32-row (K) or 8-row (V) translate of a row.
    auto kswz = [](int r) __attribute__((always_inline)) { return (r / (256 / KROW)) & (KCPR - 1); };
    auto vswz = [](int r) __attribute__((always_inline)) { return ((r / (256 / VROW)) & (VCPR / 2 - 1)) * 2; };
    // LDS row of a K stage -> key offset in the block
    auto krow_key = [](int r) __attribute__((always_inline)) { return 32 * (r >> 5) + a_row_to_key(r & 31); };

    // ---- persistent loop over this workgroup's tile pairs (heavier tile first;
    // PAIR: single tiles, p.pairs = n_tiles) ----
    const UnitRange ur = unit_range(p);
    const int T = p.n_tiles;
    for (long long u = ur.begin + ur.first; u < ur.end; u += ur.stride) {
    for (int half = 0; half < 2; ++half) {
        const int bh = (int)(u / p.pairs);
        const int pr = (int)(u - (long long)bh * p.pairs);
        const int tile = PAIR ? pr : half == 0 ? T - 1 - pr : pr;
        if (half == 1 && (PAIR || tile == T - 1 - pr))
            break;                                    // odd tile count: the middle tile is alone
        // N query rows; Nk keys; row r at key position r + qoff (qoff = 0 for
        // self-attention; otherwise a multiple of BC, so that every row of a
        // wave still lies in one BC-block of key positions)
        const int N = p.N, Nk = p.Nk, qoff = p.qoff;
        const int b = bh / p.Hq;
        const int hq = bh - b * p.Hq;
        const int hk = hq / (p.Hq / p.Hkv);
        const int tid = threadIdx.x;
        const int lane = tid & 63;
        const int w = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave index, scalar
        const int grp = w >> 2;                                   // 0: waves 0-3, 1: waves 4-7
        const int n = lane & 31;
        const int h = lane >> 5;
        const int row0 = tile * BM;
        const int wrow0 = row0 + 32 * (PAIR ? (w & 3) : w);
        const int row = wrow0 + n;

        const uint8_t* Qg = static_cast<const uint8_t*>(p.q) + (size_t)bh * N * KROW;
        const size_t kvrow0 = ((size_t)b * p.Hkv + hk) * (size_t)Nk;
        const uint8_t* Kg = static_cast<const uint8_t*>(p.k) + kvrow0 * KROW;
        const uint8_t* Vg = static_cast<const uint8_t*>(p.v) + kvrow0 * D;

        const int last_row_wg = min(row0 + BM, N) - 1;
        const int nb = CAUSAL ? (last_row_wg + qoff) / BC + 1 : (Nk + BC - 1) / BC;
        const bool wave_on = wrow0 < N;
        // every row of a wave lies in one BC-block of rows (BC is a multiple of 32)
        const int nblk_w = CAUSAL ? (min(wrow0 + 31, N - 1) + qoff) / BC + 1 : nb;
        auto jof = [&](int k) __attribute__((always_inline)) { return p.order == 0 ? k : nb - 1 - k; };
        auto valid = [&](int k) __attribute__((always_inline)) { return k >= 0 && k < nb && wave_on && jof(k) < nblk_w; };

        // ---- direct global -> LDS loads of one K / V stage (waves 0-3) ----
        // Load instruction i = wl + 4 it of a stage (wl = w & 3) writes LDS bytes
        // [1024 i, +1024): lane l fills row 4 K_RPI it + rho, rho = wl K_RPI +
        // l / KCPR, physical chunk l % KCPR, i.e. logical chunk
        // (l % KCPR) ^ kswz(rho) of key krow_key(4 K_RPI it) + krow_key(rho)
        // (4 K_RPI is a power of two >= 16, so the two key parts have disjoint
        // bits and the swizzle does not depend on it).  V likewise with
        // key = row.  Keys past the end of the sequence (only in a ragged last
        // block) read row Nk-1: they are masked to P = 0 before they can contribute.
        // The per-lane offset is taken from the block's first row, so it stays
        // below 2^32 for any number of keys.
        const int wl = w & 3;
        int k_key_l, v_key_l;
        uint32_t k_chunk_l, v_chunk_l;
        {
            const int rk = wl * K_RPI + lane / KCPR;
            k_key_l = krow_key(rk);
            k_chunk_l = (uint32_t)(((lane % KCPR) ^ kswz(rk)) * 16);
            const int rv = wl * V_RPI + lane / VCPR;
            v_key_l = rv;
            v_chunk_l = (uint32_t)(((lane % VCPR) ^ vswz(rv)) * 16);
        }
        const uint32_t k_voff = (uint32_t)k_key_l * KROW + k_chunk_l;
        const uint32_t v_voff = (uint32_t)v_key_l * VROW + v_chunk_l;
        auto load_k = [&](auto dst, int j) __attribute__((always_inline)) {
            const int t0 = j * BC;
            if (t0 + BC <= Nk) {
#pragma unroll
                for (int it = 0; it < K_NI; ++it)
                    g2lds16(Kg + (size_t)(t0 + krow_key(4 * K_RPI * it)) * KROW, k_voff,
                            lds_addr(dst) + (wl + 4 * it) * 1024);
            } else {
#pragma unroll
                for (int it = 0; it < K_NI; ++it) {
                    const int key = min(t0 + krow_key(4 * K_RPI * it) + k_key_l, Nk - 1);
                    g2lds16(Kg + (size_t)t0 * KROW, (uint32_t)(key - t0) * KROW + k_chunk_l,
                            lds_addr(dst) + (wl + 4 * it) * 1024);
                }
            }
        };
        auto load_v = [&](auto dst, int j) __attribute__((always_inline)) {
            const int t0 = j * BC;
            if (t0 + BC <= Nk) {
#pragma unroll
                for (int it = 0; it < V_NI; ++it)
                    g2lds16(Vg + (size_t)(t0 + 4 * V_RPI * it) * VROW, v_voff, lds_addr(dst) + (wl + 4 * it) * 1024);
            } else {
#pragma unroll
                for (int it = 0; it < V_NI; ++it) {
                    const int key = min(t0 + 4 * V_RPI * it + v_key_l, Nk - 1);
                    g2lds16(Vg + (size_t)t0 * VROW, (uint32_t)(key - t0) * VROW + v_chunk_l,
                            lds_addr(dst) + (wl + 4 * it) * 1024);
                }
            }
        };

        // Q^T fragments (B operand): lane (n, h) holds Q[row][16 kk + 8 h .. +8]
        // (bf16) or Q[row][64 kk + 32 h .. +32] (E4M3)
        using QFrag = std::conditional_t<QK8, i32x8, bf16x8>;
        constexpr int QSTEP = QK8 ? 64 : 32;    // bytes of a Q row per k-step
        QFrag qf[DK];
        if (row < N) {
            const uint8_t* qr = Qg + (size_t)row * KROW;
#pragma unroll
            for (int kk = 0; kk < DK; ++kk)
                qf[kk] = *reinterpret_cast<const QFrag*>(qr + QSTEP * kk + (QSTEP / 2) * h);
        } else {
#pragma unroll
            for (int kk = 0; kk < DK; ++kk)
                qf[kk] = QFrag{};
        }

        // per-lane LDS offsets.  S^T A operand of k-step kk, tile kt: LDS row
        // 32 kt + n, logical chunk 2 kk + h, i.e. (k_lane ^ (kk << 5)) + kt 32 KROW.
        // V^T operand of d-tile dt: rows (j16 >> 1) + 16 h + {0, 8, 32, 40} + 64 js,
        // logical chunk 2 dt + (n >> 4), half j16 & 1, i.e. (v_lane ^ (dt << 5)) +
        // row offset.  (The XOR only touches chunk bits; row offsets are
        // multiples of 8 rows and leave both swizzles unchanged.)
        // E4M3 K: lane (n, h) reads logical chunks 4 kk + 2 h and 4 kk + 2 h + 1.
        const uint32_t k_lane = (uint32_t)(n * KROW + (((QK8 ? 2 * h : h) ^ kswz(n)) << 4));
        const uint32_t k_lane1 = (uint32_t)(n * KROW + (((2 * h + 1) ^ kswz(n)) << 4));
        const int j16 = n & 15;                                   // lane within its 16-lane group
        const uint32_t v_lane = (uint32_t)(((j16 >> 1) + 16 * h) * VROW + (((n >> 4) | vswz(j16 >> 1)) << 4) +
                                           8 * (j16 & 1));

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
        f32x16 s[KT];                 // S^T of the block between its MFMA and VALU phases
        uint32_t pk[KT][4] = {};      // E4M3 P bytes between the VALU and the next MFMA phase
        // dynamic scale: E8M0 byte 127 + k0 - kj of each row's block, the P.V
        // MFMA's B-operand scale, which takes the block back to S units
        int pv_sb = 127;
        uint32_t cnt0 = 0, cnt1 = 0, cnt2 = 0;

        // ---- S^T = K_j Q^T (register r of tile kt: key t0 + 32 kt + 16 h + r) ----
        // The K fragments of k-step kk+2 are requested before the MFMAs of step
        // kk are issued (three rotating register sets), so LDS latency and the
        // CU-wide LDS bandwidth (shared with three other waves in this phase)
        // overlap the matrix core; sched_barrier keeps the compiler from sinking
        // the reads back next to their uses.
        // (PAIR: kst is the stage's LDS address)
        auto qk = [&](auto kst) __attribute__((always_inline)) {
            auto kfrag = [&](int kk, int kt) __attribute__((always_inline)) {
                if constexpr (QK8) {
                    const i32x4 lo = *reinterpret_cast<const i32x4*>(kst + (k_lane ^ (uint32_t)(kk << 6)) + kt * 32 * KROW);
                    const i32x4 hi = *reinterpret_cast<const i32x4*>(kst + (k_lane1 ^ (uint32_t)(kk << 6)) + kt * 32 * KROW);
                    return i32x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
                } else {
                    return *reinterpret_cast<const bf16x8*>(kst + (k_lane ^ (uint32_t)(kk << 5)) + kt * 32 * KROW);
                }
            };
            // the KT fragments of k-step kk
            auto kstep = [&](int kk, QFrag* dst) __attribute__((always_inline)) {
                if constexpr (PAIR) {
                    if constexpr (QK8) {
                        const uint32_t b0 = lds_base(kst + (lds_base(k_lane) ^ (uint32_t)(kk << 6)));
                        const uint32_t b1 = lds_base(kst + (lds_base(k_lane1) ^ (uint32_t)(kk << 6)));
#pragma unroll
                        for (int kt = 0; kt < KT; ++kt) {
                            const i32x4 lo = lds_load<i32x4>(b0 + kt * 32 * KROW);
                            const i32x4 hi = lds_load<i32x4>(b1 + kt * 32 * KROW);
                            dst[kt] = i32x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
                        }
                    } else {
                        const uint32_t b0 = lds_base(kst + (lds_base(k_lane) ^ (uint32_t)(kk << 5)));
#pragma unroll
                        for (int kt = 0; kt < KT; ++kt)
                            dst[kt] = lds_load<bf16x8>(b0 + kt * 32 * KROW);
                    }
                } else {
#pragma unroll
                    for (int kt = 0; kt < KT; ++kt)
                        dst[kt] = kfrag(kk, kt);
                }
            };
            constexpr int PF = DK >= 3 ? 2 : DK - 1;    // prefetch distance in k-steps
            QFrag a[PF + 1][KT];
#pragma unroll
            for (int kk = 0; kk < PF; ++kk)
                kstep(kk, a[kk]);
#pragma unroll
            for (int kk = 0; kk < DK; ++kk) {
                if (kk + PF < DK)
                    kstep(kk + PF, a[(kk + PF) % (PF + 1)]);
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int kt = 0; kt < KT; ++kt) {
                    const f32x16 acc = kk == 0 ? f32x16{} : s[kt];
                    if constexpr (QK8)
                        s[kt] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a[kk % (PF + 1)][kt], qf[kk], acc,
                                                                                0, 0, 0, 0, 0, 0);
                    else
                        s[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[kk % (PF + 1)][kt], qf[kk], acc, 0, 0, 0);
                }
                __builtin_amdgcn_sched_barrier(0);
            }
        };

        // ---- O^T += V_j^T P8^T ----
        // The V^T operands are read (transposed) two MFMAs ahead of their use.
        // (PAIR: vst is the stage's LDS address)
        auto pv = [&](auto vst) __attribute__((always_inline)) {
            auto vload = [&](int i) __attribute__((always_inline)) {
                const int js = i / DT, dt = i % DT;
                if constexpr (PAIR) {
                    const uint32_t va = lds_base(vst + (lds_base(v_lane) ^ (uint32_t)(dt << 5))) + 64 * js * VROW;
                    auto tr8 = [](uint32_t a) __attribute__((always_inline)) {
                        return __builtin_amdgcn_ds_read_tr8_b64_v2i32(
                            reinterpret_cast<__attribute__((address_space(3))) i32x2*>((uintptr_t)a));
                    };
                    const i32x2 r0 = tr8(va);
                    const i32x2 r1 = tr8(va + 8 * VROW);
                    const i32x2 r2 = tr8(va + 32 * VROW);
                    const i32x2 r3 = tr8(va + 40 * VROW);
                    return i32x8{r0[0], r0[1], r1[0], r1[1], r2[0], r2[1], r3[0], r3[1]};
                } else {
                    const uint8_t* va = vst + (v_lane ^ (uint32_t)(dt << 5)) + 64 * js * VROW;
                    const i32x2 r0 = lds_read_tr8(va);
                    const i32x2 r1 = lds_read_tr8(va + 8 * VROW);
                    const i32x2 r2 = lds_read_tr8(va + 32 * VROW);
                    const i32x2 r3 = lds_read_tr8(va + 40 * VROW);
                    return i32x8{r0[0], r0[1], r1[0], r1[1], r2[0], r2[1], r3[0], r3[1]};
                }
            };
            constexpr int NM = PVS * DT;                 // FP8 MFMAs per block
            constexpr int PF = NM >= 3 ? 2 : NM - 1;
            i32x8 av[PF + 1];
#pragma unroll
            for (int i = 0; i < PF; ++i)
                av[i] = vload(i);
#pragma unroll
            for (int i = 0; i < NM; ++i) {
                const int js = i / DT, dt = i % DT;
                if (i + PF < NM)
                    av[(i + PF) % (PF + 1)] = vload(i + PF);
                i32x8 bop;
#pragma unroll
                for (int q4 = 0; q4 < 4; ++q4) {
                    bop[q4] = (int)pk[2 * js][q4];
                    bop[4 + q4] = (int)pk[2 * js + 1][q4];
                }
                __builtin_amdgcn_sched_barrier(0);
                if constexpr (SCALE == kScaleDynamic)
                    o[dt] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av[i % (PF + 1)], bop, o[dt], 0, 0, 0,
                                                                            127, 0, pv_sb);
                else
                    o[dt] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av[i % (PF + 1)], bop, o[dt], 0, 0, 0,
                                                                            0, 0, 0);
                __builtin_amdgcn_sched_barrier(0);
            }
        };

        // ---- running max, alpha, P, l (pre-cast), E4M3 cast, rescale of O ----
        auto softmax = [&](int j) __attribute__((always_inline)) {
            const int t0 = j * BC;
            if ((CAUSAL && j == nblk_w - 1) || t0 + BC > Nk) {
                // key t0 + 32 kt + 16 h + r is valid iff 32 kt + r <= lim; masked
                // scores become -inf through a sign-mask bit select (no compares)
                const int lim = (CAUSAL ? min(row + qoff, Nk - 1) : Nk - 1) - t0 - 16 * h;
#pragma unroll
                for (int kt = 0; kt < KT; ++kt)
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const uint32_t m = (uint32_t)((lim - (32 * kt + r)) >> 31);
                        const float sv = s[kt][r];
                        const uint32_t x = __float_as_uint(sv);
                        s[kt][r] = __uint_as_float((x & ~m) | (0xFF800000u & m));
                    }
            }
            // row maximum: one independent chain per 32-key tile, then the tiles,
            // then the two lane halves (a maximum is exact in any order)
            float mk[KT];
#pragma unroll
            for (int kt = 0; kt < KT; ++kt) {
                float a = s[kt][0];
#pragma unroll
                for (int r = 1; r < 16; ++r)
                    a = fmax_f(a, s[kt][r]);
                mk[kt] = a;
            }
            float mx = mk[0];
#pragma unroll
            for (int kt = 1; kt < KT; ++kt)
                mx = fmax_f(mx, mk[kt]);
            mx = halves_max(mx);
            // PAIR: the running maximum after the previous block of the visit
            // (the partner's, or an earlier one if the partner skipped its
            // blocks) comes from LDS; alpha still takes this wave's own (O, l)
            // from its last block to the new maximum
            float m_prev = m_run;
            if constexpr (PAIR)
                m_prev = mslot[w & 3][n];
            const float m_new = fmax_f(m_prev, mx);
            const float mc_new = m_new * c;
            const float alpha = __builtin_amdgcn_exp2f(mc_run - mc_new);
            const float nmc = -mc_new;
            if (COUNT && p.gap_hist && h == 0 && row < N)
                record_gap(p, bh, j, mx, c, nmc);
            // Dynamic P-scale (Limitations and Future Work, read as: the
            // block's largest P lands in (S/2, S]): kj = k0 + clamp(floor(-xmax),
            // 0, 126 - k0), xmax = fma(block max, c, -mc).  The convert scales
            // by 2^kj (scale operand 2^-kj) and P.V by 2^(k0 - kj).
            float cvt_scale = inv_S;
            if constexpr (SCALE == kScaleDynamic) {
                const float xmax = __builtin_fmaf(mx, c, nmc);
                const float f = __builtin_fminf(__builtin_fmaxf(__builtin_floorf(-xmax), 0.f),
                                                (float)(126 - p.k0));
                const int kj = p.k0 + (int)f;
                cvt_scale = __uint_as_float((uint32_t)(127 - kj) << 23);
                pv_sb = 127 + p.k0 - kj;
            }
            // The rest is organised in stages so that no instruction waits on the
            // result of the one just before it (this phase runs alone on its
            // SIMD's vector ALU while the partner wave drives the matrix core):
            // (1) x = fma(D, c, -mc) for all keys, in place;
            // (2) P = exp2(x) for all keys, in place, interleaved with the rescale
            //     of O (independent work for the vector ALU while exp2 is in flight);
            // (3) l from the pre-cast P (one partial sum per tile), E4M3 cast.
#pragma unroll
            for (int kt = 0; kt < KT; ++kt)
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    s[kt][r] = __builtin_fmaf(s[kt][r], c, nmc);
            __builtin_amdgcn_sched_barrier(0);
            // rescale O before this block's P.V; skipped when no row of the wave
            // moved its maximum (alpha is then exactly 1)
            const bool rescale = __ballot(alpha != 1.0f) != 0;
            if (rescale) {
#pragma unroll
                for (int t = 0; t < DT; ++t)
#pragma unroll
                    for (int r = 0; r < 16; ++r)
                        o[t][r] *= alpha;
            }
            {
#pragma unroll
                for (int kt = 0; kt < KT; ++kt)
#pragma unroll
                    for (int r = 0; r < 16; ++r)
                        s[kt][r] = __builtin_amdgcn_exp2f(s[kt][r]);
            }
            __builtin_amdgcn_sched_barrier(0);
            uint32_t bz = 0;   // zero codes of this block (valid rows and keys)
            // keys of the sink's block, the diagonal block and a ragged last
            // block need a validity and category mask per word
            const bool slow_count = j == 0 || (CAUSAL && j == nblk_w - 1) || t0 + BC > Nk;
            float lpart[KT];
#pragma unroll
            for (int kt = 0; kt < KT; ++kt) {
                float l0 = s[kt][0] + s[kt][1], l1 = s[kt][2] + s[kt][3];
#pragma unroll
                for (int r = 4; r < 16; r += 4) {
                    l0 += s[kt][r] + s[kt][r + 1];
                    l1 += s[kt][r + 2] + s[kt][r + 3];
                }
                lpart[kt] = l0 + l1;
            }
#pragma unroll
            for (int kt = 0; kt < KT; ++kt) {
#pragma unroll
                for (int r4 = 0; r4 < 4; ++r4) {
                    const float p0 = s[kt][4 * r4 + 0], p1 = s[kt][4 * r4 + 1];
                    const float p2 = s[kt][4 * r4 + 2], p3 = s[kt][4 * r4 + 3];
                    uint32_t word;
                    // The first convert writes the low half of the word, the second
                    // the high half; the stale bytes of the previous block that the
                    // word starts from are all overwritten (no zeroing needed).
                    if constexpr (SCALE != kScaleAny) {
                        s16x2 lo = __builtin_bit_cast(s16x2, pk[kt][r4]);
                        lo = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(lo, p0, p1, cvt_scale, false);
                        lo = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(lo, p2, p3, cvt_scale, true);
                        word = __builtin_bit_cast(uint32_t, lo);
                    } else {
                        const float y0 = __builtin_fminf(p0 * S, 448.f);
                        const float y1 = __builtin_fminf(p1 * S, 448.f);
                        const float y2 = __builtin_fminf(p2 * S, 448.f);
                        const float y3 = __builtin_fminf(p3 * S, 448.f);
                        int wv = __builtin_amdgcn_cvt_pk_fp8_f32(y0, y1, (int)pk[kt][r4], false);
                        wv = __builtin_amdgcn_cvt_pk_fp8_f32(y2, y3, wv, true);
                        word = (uint32_t)wv;
                    }
                    pk[kt][r4] = word;
                }
            }
            // every key of a block past the sink's, off the diagonal and inside
            // the keys is valid and in category 2: count its zero codes by word
            if (COUNT && slow_count) {
                // byte i of word (kt, r4) holds key t0 + o + i, o = 32 kt + 16 h + 4 r4;
                // it is valid iff o + i <= lim, and a sink key iff o + i < ns
                const int lim = (CAUSAL ? min(row + qoff, Nk - 1) : Nk - 1) - t0;
                const int ns = j == 0 ? p.n_sink : 0;
                auto low_bytes = [](int n) __attribute__((always_inline)) {
                    const int c = min(max(n, 0), 4);
                    return (uint32_t)((1ull << (8 * c)) - 1);
                };
                uint32_t z0 = 0, zn = 0;
#pragma unroll
                for (int kt = 0; kt < KT; ++kt)
#pragma unroll
                    for (int r4 = 0; r4 < 4; ++r4) {
                        const int o = 32 * kt + 16 * h + 4 * r4;
                        const uint32_t valid = low_bytes(lim - o + 1);
                        const uint32_t sink = low_bytes(ns - o);
                        const uint32_t wd = pk[kt][r4];
                        // invalid or other-category bytes are forced non-zero
                        z0 += zero_codes(wd | ~(valid & sink));
                        zn += zero_codes(wd | ~(valid & ~sink));
                    }
                if (j > 0) {
                    cnt2 += zn;
                } else {
                    cnt0 += z0;
                    cnt1 += zn;
                }
                bz += row < N ? z0 + zn : 0u;
            }
            if (COUNT && !slow_count) {
                uint32_t zc = 0;
#pragma unroll
                for (int kt = 0; kt < KT; ++kt)
#pragma unroll
                    for (int r4 = 0; r4 < 4; ++r4)
                        zc += zero_codes(pk[kt][r4]);
                cnt2 += zc;
                bz += row < N ? zc : 0u;
            }
            if (COUNT && p.blk_zero)
                record_block_zeros(p, bh, j, bz);
            float lsum = lpart[0];
#pragma unroll
            for (int kt = 1; kt < KT; ++kt)
                lsum += lpart[kt];
            ell = alpha * ell + lsum;
            m_run = m_new;
            mc_run = mc_new;
            if constexpr (PAIR)
                mslot[w & 3][n] = m_new;
        };

        // ---- prologue: K of the first block into stage 0 ----
        if constexpr (PAIR) {
            if (grp == 0) {
                load_k(Kst, jof(0));
                mslot[w][n] = -INFINITY;
            }
        } else {
            if (grp == 0)
                load_k(Sst, jof(0));
        }
        // Q fragments and the first K stage are complete after this point; the
        // compiler sees the wait (it tracks no outstanding loads in the loop)
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        // Both groups run the same program -- per block k an MFMA phase (P.V of
        // block k-1, S^T of block k) and a VALU phase (softmax of block k), each
        // closed by a workgroup barrier -- but group 1 first passes one extra
        // barrier, so it runs one phase behind group 0: while one wave of a SIMD
        // is in its MFMA phase the other is in its softmax phase.  Group 0 issues
        // the loads of K_{k+1} and V_k at the start of its MFMA phase k; they are
        // first read two phases later.  Stage parity is k % 2 (the loop is
        // unrolled twice so every LDS access names its stage statically).
        if (grp == 1)
            __syncthreads();
        if constexpr (PAIR) {
            // PAIR: group g processes the blocks at visit positions k = 2 i + g.
            // Its MFMA phase i (P.V of its previous block k - 2, S^T of block k)
            // is phase k of the workgroup and its softmax of block k phase k + 1,
            // so block k's softmax follows block k - 1's (the partner's) with a
            // barrier between them.  K_k is read only in phase k and V_k only in
            // phase k + 2, both from stage k % 2 = g: a group reads its own
            // stages and, at the start of its MFMA phase k, copies K_{k+1} and
            // V_{k-1} into the other group's (last read in phase k - 1), waiting
            // for them at the end of the phase.  (A third stage, copied two
            // phases ahead from either side of the phase, measured slower.)
            const uint32_t k_own = lds_addr(Kst) + (uint32_t)(grp * K_BYTES);
            const uint32_t k_oth = lds_addr(Kst) + (uint32_t)((1 - grp) * K_BYTES);
            const uint32_t v_own = lds_addr(Vst) + (uint32_t)(grp * V_BYTES);
            const uint32_t v_oth = lds_addr(Vst) + (uint32_t)((1 - grp) * V_BYTES);
            auto pair_iteration = [&](int i) __attribute__((always_inline)) {
                const int kq = 2 * i + grp;
                if (kq + 1 < nb)
                    load_k(k_oth, jof(kq + 1));
                if (kq >= 1 && kq - 1 < nb)
                    load_v(v_oth, jof(kq - 1));
                __builtin_amdgcn_sched_barrier(0);
                __builtin_amdgcn_s_setprio(1);
                __builtin_amdgcn_sched_barrier(0);
                if (valid(kq - 2))
                    pv(v_own);
                if (valid(kq))
                    qk(k_own);
                __builtin_amdgcn_sched_barrier(0);
                __builtin_amdgcn_s_setprio(0);
                __builtin_amdgcn_sched_barrier(0);
                wait_loads();
                __syncthreads();
                if (valid(kq))
                    softmax(jof(kq));
                __syncthreads();
            };
            // both groups pass the same number of barriers; the last P.V of
            // a group comes two phases after its last block
            const int I = (nb + 3) / 2;
            for (int i = 0; i < I; ++i)
                pair_iteration(i);
        } else {
            auto iteration = [&](int k, uint8_t* k_cur, uint8_t* k_nxt, uint8_t* v_cur, uint8_t* v_prv)
                __attribute__((always_inline)) {
                if (grp == 0) {
                    if (k + 1 < nb)
                        load_k(k_nxt, jof(k + 1));
                    if (k < nb)
                        load_v(v_cur, jof(k));
                }
                // the wave in its MFMA phase takes issue priority over its SIMD
                // partner in the VALU phase, so the matrix core is fed first
                __builtin_amdgcn_sched_barrier(0);
                __builtin_amdgcn_s_setprio(1);
                __builtin_amdgcn_sched_barrier(0);
                if (valid(k - 1))
                    pv(v_prv);
                if (valid(k))
                    qk(k_cur);
                __builtin_amdgcn_sched_barrier(0);
                __builtin_amdgcn_s_setprio(0);
                __builtin_amdgcn_sched_barrier(0);
                __syncthreads();
                if (valid(k))
                    softmax(jof(k));
                // the stage loads issued in the MFMA phase must land before the
                // barrier that hands them to the next MFMA phase
                if (grp == 0)
                    wait_loads();
                __syncthreads();
            };
            uint8_t* const Ks0 = Sst;
            uint8_t* const Ks1 = Sst + K_BYTES;
            uint8_t* const Vs0 = Sst + 2 * K_BYTES;
            uint8_t* const Vs1 = Sst + 2 * K_BYTES + V_BYTES;
            for (int k = 0; k <= nb; k += 2) {
                iteration(k, Ks0, Ks1, Vs0, Vs1);
                if (k + 1 <= nb)
                    iteration(k + 1, Ks1, Ks0, Vs1, Vs0);
            }
        }
        if (grp == 0)
            __syncthreads();

        if constexpr (PAIR) {
            // The row group's two partials.  This wave's (O, l) is at the
            // maximum of its own last block; bring it to the rows' final
            // maximum (the slot after the last block of the visit), then
            // group 1 hands its partial to group 0 through LDS: O through K
            // stage 1 in rounds of XR 16-byte pieces per lane, l and the
            // counts through V stage 0.  K stage 0 is left alone (the next
            // tile's first K block lands there before its first barrier).  (Rows whose
            // waves saw no block keep -inf: factor 1.)
            const float mc_f = mslot[w & 3][n] * c;
            const float a = mc_run == mc_f ? 1.0f : __builtin_amdgcn_exp2f(mc_run - mc_f);
            ell *= a;
#pragma unroll
            for (int dt = 0; dt < DT; ++dt)
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    o[dt][r] *= a;
            mc_run = mc_f;
            constexpr int XR = K_BYTES / 4096 < 4 * DT ? K_BYTES / 4096 : 4 * DT;   // pieces per round
            static_assert(XR >= 1 && (4 * DT) % XR == 0 && V_BYTES >= 4096, "handoff layout");
            f32x4* const xw = reinterpret_cast<f32x4*>(Kst + K_BYTES) + ((w & 3) * 64 + lane) * XR;
            float* const xsw = reinterpret_cast<float*>(Vst) + ((w & 3) * 64 + lane) * 4;
            if (grp == 1) {
                xsw[0] = ell;
                xsw[1] = __uint_as_float(cnt0);
                xsw[2] = __uint_as_float(cnt1);
                xsw[3] = __uint_as_float(cnt2);
            }
#pragma unroll
            for (int r0 = 0; r0 < 4 * DT; r0 += XR) {
                if (grp == 1) {
#pragma unroll
                    for (int x = 0; x < XR; ++x) {
                        const int dt = (r0 + x) / 4, r4 = (r0 + x) % 4;
                        xw[x] = f32x4{o[dt][4 * r4], o[dt][4 * r4 + 1], o[dt][4 * r4 + 2], o[dt][4 * r4 + 3]};
                    }
                }
                __syncthreads();
                if (grp == 0) {
#pragma unroll
                    for (int x = 0; x < XR; ++x) {
                        const int dt = (r0 + x) / 4, r4 = (r0 + x) % 4;
                        const f32x4 x4 = xw[x];
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            o[dt][4 * r4 + e] += x4[e];
                    }
                    if (r0 == 0) {
                        ell += xsw[0];
                        cnt0 += __float_as_uint(xsw[1]);
                        cnt1 += __float_as_uint(xsw[2]);
                        cnt2 += __float_as_uint(xsw[3]);
                    }
                }
                __syncthreads();
            }
        }

        if (!wave_on || (PAIR && grp == 1))
            continue;
        const float ell_row = ell + other_half(ell);
        if (COUNT) {
            cnt0 += other_half_u32(cnt0);
            cnt1 += other_half_u32(cnt1);
            cnt2 += other_half_u32(cnt2);
        }
        // Output through LDS (256-row schedule, d = 128): each wave stages its
        // 32 rows x 32 columns per round (4 KB, wave w at K_BYTES + 4096 w, past
        // stage K 0, the only stage the next tile writes before its first
        // barrier) and stores 8 whole 128-byte row segments per instruction,
        // instead of 32 rows x 32 bytes straight from the accumulator layout.
        constexpr bool STAGED_OUT = !PAIR && D == 128 && K_BYTES + V_BYTES >= 8 * 4096;
        if constexpr (STAGED_OUT) {
            if (p.out) {
                const float inv = p.v_descale / (S * ell_row);
                // per-lane LDS addresses, materialised here (not hoisted out of
                // the tile loop): write chunk c = 2 r4 + h of row n at
                // 16 (c ^ (n & 7)) = wa ^ 32 r4; read row 8 i + rr, chunk cc at ra + 1024 i
                const uint32_t base_w = lds_addr(Sst) + K_BYTES + 4096u * (uint32_t)w;
                const uint32_t x = (uint32_t)n & 7u;
                const uint32_t wa = lds_base(base_w + 128u * (uint32_t)n + 16u * ((uint32_t)h ^ (x & 1u)) +
                                             32u * (x >> 1));
                const uint32_t rr = (uint32_t)lane >> 3, cc = (uint32_t)lane & 7u;
                const uint32_t ra = lds_base(base_w + 128u * rr + 16u * (cc ^ rr));
                float* const orow0 = p.out + ((size_t)bh * N + wrow0 + rr) * D + 4 * cc;
#pragma unroll
                for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
                    for (int r4 = 0; r4 < 4; ++r4) {
                        f32x4 v4;
                        v4[0] = o[dt][4 * r4 + 0] * inv;
                        v4[1] = o[dt][4 * r4 + 1] * inv;
                        v4[2] = o[dt][4 * r4 + 2] * inv;
                        v4[3] = o[dt][4 * r4 + 3] * inv;
                        *reinterpret_cast<__attribute__((address_space(3))) f32x4*>((uintptr_t)(wa ^ (32u * r4))) = v4;
                    }
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const f32x4 v4 = lds_load<f32x4>(ra + 1024u * i);
                        if (wrow0 + 8 * i + (int)rr < N)
                            *reinterpret_cast<f32x4*>(orow0 + (size_t)8 * i * D + 32 * dt) = v4;
                    }
                }
            }
        }
        if (row < N) {
            const size_t flat = (size_t)bh * N + row;
            if (!STAGED_OUT && p.out) {
                const float inv = p.v_descale / (S * ell_row);
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
    }  // tile of the pair
    }  // unit
}

}  // namespace attn
