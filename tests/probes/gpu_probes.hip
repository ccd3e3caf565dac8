// Hardware probes for the GPU tests (test infrastructure, not part of the
// library).  Each probe runs one gfx950 instruction the attention kernels rely
// on over caller-chosen inputs, so the tests can compare it with the CPU
// oracle or with exact host arithmetic:
//   - v_cvt_pk_fp8_f32 and v_cvt_scalef32_pk_fp8_f32 (the E4M3 P-cast),
//   - v_exp_f32 (exp2 in the fast kernels),
//   - the operand/accumulator lane layouts of the three MFMA shapes used,
//   - the per-lane E8M0 operand scales of the block-scaled FP8 MFMA and the
//     per-lane scale of the scaled convert (the dynamic P-scale),
//   - the chip-wide issue rate of v_exp_f32 (the exp2 peak the attention
//     kernels are measured against),
//   - the LDS read rate of one CU (ds_read_b128 and the transposing
//     ds_read_b64_tr_b8, the two reads of the MFMA phase), alone and while
//     other waves of the workgroup copy global memory into LDS with
//     global_load_lds_dwordx4 (the stage copies),
//   - how the matrix core and the vector ALU of one SIMD overlap: the matrix
//     and the vector work of one wave and key block, each alone, split over
//     two waves of a SIMD (the fast kernel's ping-pong) or interleaved in one
//     wave per SIMD, and what each MFMA shape costs the vector wave.
// Every kernel bounds-checks its index against n.
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(8 * sizeof(int)))) int i32x8;
typedef __attribute__((__vector_size__(2 * sizeof(short)))) short s16x2;
typedef __attribute__((__vector_size__(4 * sizeof(int)))) int i32x4;
typedef __attribute__((__vector_size__(2 * sizeof(int)))) int i32x2;

__global__ void k_cvt_range(uint32_t lo, int64_t n, uint8_t* out)
{
    const int64_t i = 2 * ((int64_t)blockIdx.x * blockDim.x + threadIdx.x);
    if (i >= n)
        return;
    const float x0 = __builtin_bit_cast(float, (uint32_t)(lo + i));
    const float x1 = (i + 1 < n) ? __builtin_bit_cast(float, (uint32_t)(lo + i + 1)) : 0.f;
    const int w = __builtin_amdgcn_cvt_pk_fp8_f32(x0, x1, 0, false);
    out[i] = (uint8_t)(w & 0xFF);
    if (i + 1 < n)
        out[i + 1] = (uint8_t)((w >> 8) & 0xFF);
}

__global__ void k_cvt_list(const float* x, int64_t n, uint8_t* out, float scale, int scaled, int hi)
{
    const int64_t i = 2 * ((int64_t)blockIdx.x * blockDim.x + threadIdx.x);
    if (i >= n)
        return;
    const float x0 = x[i];
    const float x1 = (i + 1 < n) ? x[i + 1] : 0.f;
    uint32_t w;
    s16x2 z = {0, 0};
    if (scaled && hi)
        w = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(z, x0, x1, scale, true));
    else if (scaled)
        w = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(z, x0, x1, scale, false));
    else if (hi)
        w = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(x0, x1, 0, true);
    else
        w = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(x0, x1, 0, false);
    if (hi)
        w >>= 16;
    out[i] = (uint8_t)(w & 0xFF);
    if (i + 1 < n)
        out[i + 1] = (uint8_t)((w >> 8) & 0xFF);
}

__global__ void k_exp2(const float* x, int64_t n, float* out)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n)
        out[i] = __builtin_amdgcn_exp2f(x[i]);
}

// v_exp_f32 throughput: every lane runs 16 independent chains x <- exp2(-x)
// (which stays in [0.5, 1]) for `iters` rounds; 256-thread workgroups, one
// result per lane written so the work is kept.
__global__ void __launch_bounds__(256) k_exp2_rate(int iters, float* out)
{
    float x[16];
#pragma unroll
    for (int i = 0; i < 16; ++i)
        x[i] = 0.5f + 0.03125f * (float)i + 1e-6f * (float)threadIdx.x;
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int i = 0; i < 16; ++i)
            x[i] = __builtin_amdgcn_exp2f(-x[i]);
    }
    float acc = 0.f;
#pragma unroll
    for (int i = 0; i < 16; ++i)
        acc += x[i];
    out[(int64_t)blockIdx.x * 256 + threadIdx.x] = acc;
}

// LDS read rate.  One workgroup of 8 waves per CU.  Reader waves issue
// rounds of 8 independent reads (mode bit 0: 0 = ds_read_b128, 1 KB per wave
// instruction; 1 = ds_read_b64_tr_b8, 512 B) over their own 8 KB of LDS, then
// wait for them; cycles[wg * 8 + wave] gets the s_memtime cycles of the read
// loop.  readers: waves 0..readers-1 read.  copiers: waves 8-copiers..7 copy
// 1 KB per instruction from src (64 KB, L2-resident after the first round)
// into a separate 16 KB of LDS with global_load_lds_dwordx4, keeping at most
// 8 copies in flight, for as many rounds as the readers run (iters * 8
// instructions); a wave is never both.  sink keeps the reads alive.
__global__ void __launch_bounds__(512) k_lds_rate(int iters, int mode, int readers, int copiers,
                                                   const uint8_t* src, unsigned long long* cycles,
                                                   uint32_t* sink)
{
    __shared__ __attribute__((aligned(1024))) uint32_t buf[16384];    // 64 KB: 8 KB per reader wave
    __shared__ __attribute__((aligned(1024))) uint8_t cbuf[32768];    // copy target (16 KB used; 96 KB in all: one workgroup per CU)
    for (int i = threadIdx.x; i < 16384; i += 512)
        buf[i] = (uint32_t)i * 2654435761u;
    __syncthreads();
    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    uint32_t acc = 0;
    unsigned long long t0 = 0, t1 = 0;
    if (w < readers) {
        const uint32_t a = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) uint32_t*)(buf + w * 2048) +
                           (mode ? 8u : 16u) * (uint32_t)lane;
        asm volatile("s_memtime %0\n\ts_waitcnt lgkmcnt(0)" : "=s"(t0) :: "memory");
        for (int it = 0; it < iters; ++it) {
            if (mode == 0) {
                i32x4 r0, r1, r2, r3, r4, r5, r6, r7;
                asm volatile(
                    "ds_read_b128 %0, %8\n\tds_read_b128 %1, %8 offset:1024\n\t"
                    "ds_read_b128 %2, %8 offset:2048\n\tds_read_b128 %3, %8 offset:3072\n\t"
                    "ds_read_b128 %4, %8 offset:4096\n\tds_read_b128 %5, %8 offset:5120\n\t"
                    "ds_read_b128 %6, %8 offset:6144\n\tds_read_b128 %7, %8 offset:7168\n\t"
                    "s_waitcnt lgkmcnt(0)"
                    : "=v"(r0), "=v"(r1), "=v"(r2), "=v"(r3), "=v"(r4), "=v"(r5), "=v"(r6), "=v"(r7)
                    : "v"(a) : "memory");
                acc ^= (uint32_t)(r0[0] ^ r1[1] ^ r2[2] ^ r3[3] ^ r4[0] ^ r5[1] ^ r6[2] ^ r7[3]);
            } else {
                i32x2 r0, r1, r2, r3, r4, r5, r6, r7;
                asm volatile(
                    "ds_read_b64_tr_b8 %0, %8\n\tds_read_b64_tr_b8 %1, %8 offset:512\n\t"
                    "ds_read_b64_tr_b8 %2, %8 offset:1024\n\tds_read_b64_tr_b8 %3, %8 offset:1536\n\t"
                    "ds_read_b64_tr_b8 %4, %8 offset:2048\n\tds_read_b64_tr_b8 %5, %8 offset:2560\n\t"
                    "ds_read_b64_tr_b8 %6, %8 offset:3072\n\tds_read_b64_tr_b8 %7, %8 offset:3584\n\t"
                    "s_waitcnt lgkmcnt(0)"
                    : "=v"(r0), "=v"(r1), "=v"(r2), "=v"(r3), "=v"(r4), "=v"(r5), "=v"(r6), "=v"(r7)
                    : "v"(a) : "memory");
                acc ^= (uint32_t)(r0[0] ^ r1[1] ^ r2[0] ^ r3[1] ^ r4[0] ^ r5[1] ^ r6[0] ^ r7[1]);
            }
        }
        asm volatile("s_waitcnt lgkmcnt(0)\n\ts_memtime %0\n\ts_waitcnt lgkmcnt(0)" : "=s"(t1) :: "memory");
    } else if (w >= 8 - copiers) {
        // copy instruction i: 1 KB from src + 1024 * (i % 64), lane l -> +16 l;
        // LDS cbuf + 1024 * (i % 16)
        const uint32_t lds0 = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) uint8_t*)cbuf;
        const uint32_t voff = 16u * (uint32_t)lane;
        asm volatile("s_memtime %0\n\ts_waitcnt lgkmcnt(0)" : "=s"(t0) :: "memory");
        for (int i = 0; i < iters * 8; ++i) {
            const uint8_t* base = src + 1024 * (i & 63);
            const uint32_t m0 = lds0 + 1024u * (uint32_t)(i & 15);
            asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2\n\ts_waitcnt vmcnt(8)"
                         :
                         : "s"(__builtin_amdgcn_readfirstlane(m0)), "v"(voff), "s"(base)
                         : "memory");
        }
        asm volatile("s_waitcnt vmcnt(0)\n\ts_memtime %0\n\ts_waitcnt lgkmcnt(0)" : "=s"(t1) :: "memory");
    }
    if (lane == 0)
        cycles[blockIdx.x * 8 + w] = t1 - t0;
    sink[blockIdx.x * 512 + threadIdx.x] = acc;
}

// One wave.  A: 32x16 bf16 (row-major), B: 16x32 bf16, D: 32x32 f32.
// Assumed layout: lane (m = l%32, h = l/32) holds A[m][8h..8h+7] and
// B[8h..8h+7][m]; accumulator register r is D[8(r/4) + 4h + r%4][l%32].
__global__ void k_mfma_bf16(const uint16_t* A, const uint16_t* B, float* D)
{
    const int l = threadIdx.x;
    if (l >= 64)
        return;
    const int m = l & 31, h = l >> 5;
    bf16x8 a, b;
    for (int i = 0; i < 8; ++i) {
        a[i] = __builtin_bit_cast(__bf16, A[m * 16 + 8 * h + i]);
        b[i] = __builtin_bit_cast(__bf16, B[(8 * h + i) * 32 + m]);
    }
    f32x16 acc = {};
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc, 0, 0, 0);
    for (int r = 0; r < 16; ++r)
        D[(8 * (r / 4) + 4 * h + (r % 4)) * 32 + m] = acc[r];
}

// One wave.  A: 32x64 E4M3 bytes, B: 64x32 E4M3 bytes, D: 32x32 f32.
// Assumed: lane (m, h) holds A[m][32h .. 32h+31] and B[32h .. 32h+31][m].
__global__ void k_mfma_fp8(const uint8_t* A, const uint8_t* B, float* D)
{
    const int l = threadIdx.x;
    if (l >= 64)
        return;
    const int m = l & 31, h = l >> 5;
    i32x8 a, b;
    for (int q = 0; q < 8; ++q) {
        uint32_t wa = 0, wb = 0;
        for (int e = 0; e < 4; ++e) {
            const int kk = 32 * h + 4 * q + e;
            wa |= (uint32_t)A[m * 64 + kk] << (8 * e);
            wb |= (uint32_t)B[kk * 32 + m] << (8 * e);
        }
        a[q] = (int)wa;
        b[q] = (int)wb;
    }
    f32x16 acc = {};
    acc = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, acc, 0, 0, 0, 0, 0, 0);
    for (int r = 0; r < 16; ++r)
        D[(8 * (r / 4) + 4 * h + (r % 4)) * 32 + m] = acc[r];
}

// One wave, the block-scaled FP8 MFMA.  As k_mfma_fp8, plus one E8M0 scale
// byte per lane for A (sa[l]) and for B (sb[l]), passed in byte 0 of the
// scale operands.  Assumed: lane (m, h)'s byte scales the 32 elements it
// supplies, A[m][32h .. 32h+31] and B[32h .. 32h+31][m], by 2^(byte - 127).
__global__ void k_mfma_fp8_scaled(const uint8_t* A, const uint8_t* B, const uint8_t* sa,
                                  const uint8_t* sb, float* D)
{
    const int l = threadIdx.x;
    if (l >= 64)
        return;
    const int m = l & 31, h = l >> 5;
    i32x8 a, b;
    for (int q = 0; q < 8; ++q) {
        uint32_t wa = 0, wb = 0;
        for (int e = 0; e < 4; ++e) {
            const int kk = 32 * h + 4 * q + e;
            wa |= (uint32_t)A[m * 64 + kk] << (8 * e);
            wb |= (uint32_t)B[kk * 32 + m] << (8 * e);
        }
        a[q] = (int)wa;
        b[q] = (int)wb;
    }
    f32x16 acc = {};
    acc = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, acc, 0, 0, 0, (int)sa[l], 0, (int)sb[l]);
    for (int r = 0; r < 16; ++r)
        D[(8 * (r / 4) + 4 * h + (r % 4)) * 32 + m] = acc[r];
}

// The scaled convert with a per-element scale: out = cvt(x[i] / scale[i]) pairs.
__global__ void k_cvt_scaled_vec(const float* x, const float* scale, int64_t n, uint8_t* out)
{
    const int64_t i = 2 * ((int64_t)blockIdx.x * blockDim.x + threadIdx.x);
    if (i + 1 >= n)
        return;
    s16x2 z = {0, 0};
    // both elements of a pair share the scale of the first
    const uint32_t w = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(z, x[i], x[i + 1], scale[i], false));
    out[i] = (uint8_t)(w & 0xFF);
    out[i + 1] = (uint8_t)((w >> 8) & 0xFF);
}

// One wave.  A: 32x2 f32, B: 2x32 f32, D: 32x32 f32.  Lane (m, h): A[m][h], B[h][m].
__global__ void k_mfma_f32(const float* A, const float* B, float* D)
{
    const int l = threadIdx.x;
    if (l >= 64)
        return;
    const int m = l & 31, h = l >> 5;
    f32x16 acc = {};
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(A[m * 2 + h], B[h * 32 + m], acc, 0, 0, 0);
    for (int r = 0; r < 16; ++r)
        D[(8 * (r / 4) + 4 * h + (r % 4)) * 32 + m] = acc[r];
}

static int grid_for(int64_t items, int per_block)
{
    return (int)((items + per_block - 1) / per_block);
}

// ---- co-execution of the matrix core and the vector ALU ----
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
// Matrix streams, each 1536 matrix-core cycles at the documented rates.
// pattern 0: one wave's matrix work per 128-key block of the fast kernel
// (d = 128, bf16 scores): 32 bf16 32x32x16 MFMAs (S^T) and 8 FP8 32x32x64
// MFMAs (P.V); 1: 24 FP8 32x32x64; 2: 48 bf16 32x32x16; 3: 96 bf16 16x16x32
// (four accumulators in rotation in every pattern)
template <int PAT>
__device__ __forceinline__ void coexec_mfma(f32x16 (&acc)[4], f32x16 (&o)[4], f32x4 (&q)[4], bf16x8 a, bf16x8 b,
                                            i32x8 a8, i32x8 b8)
{
    if constexpr (PAT == 0) {
#pragma unroll
        for (int kk = 0; kk < 8; ++kk)
#pragma unroll
            for (int kt = 0; kt < 4; ++kt)
                acc[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[kt], 0, 0, 0);
#pragma unroll
        for (int i = 0; i < 8; ++i)
            o[i & 3] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a8, b8, o[i & 3], 0, 0, 0, 0, 0, 0);
    } else if constexpr (PAT == 1) {
#pragma unroll
        for (int i = 0; i < 24; ++i)
            o[i & 3] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a8, b8, o[i & 3], 0, 0, 0, 0, 0, 0);
    } else if constexpr (PAT == 2) {
#pragma unroll
        for (int i = 0; i < 48; ++i)
            acc[i & 3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[i & 3], 0, 0, 0);
    } else {
#pragma unroll
        for (int i = 0; i < 96; ++i)
            q[i & 3] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, q[i & 3], 0, 0, 0);
    }
}

// Vector stream, the instruction mix of the softmax of one wave and block:
// a maximum over 64 values (v_max3 pairs), 64 FMAs, 64 exp2, 64 adds (the
// row sum), 32 scaled E4M3 pair converts and 64 multiplies (the rescale of O).
// Every value feeds the next iteration, so no work can be hoisted or dropped.
__device__ __forceinline__ void coexec_rescale(float (&ov)[64], float alpha)
{
#pragma unroll
    for (int i = 0; i < 64; ++i)
        ov[i] *= alpha;
}
__device__ __forceinline__ void coexec_rescale(f32x16 (&ov)[4], float alpha)
{
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r)
            ov[i][r] *= alpha;
}
template <typename OV>
__device__ __forceinline__ void coexec_valu(float (&x)[64], OV& ov, uint32_t (&pk)[16], float& l, float& mc)
{
    float mx = x[0];
#pragma unroll
    for (int i = 1; i < 63; i += 2)
        mx = __builtin_fmaxf(__builtin_fmaxf(mx, x[i]), x[i + 1]);
    mx = __builtin_fmaxf(mx, x[63]);
    const float alpha = __builtin_amdgcn_exp2f(mc - mx);
    mc = mx;
#pragma unroll
    for (int i = 0; i < 64; ++i)
        x[i] = __builtin_fmaf(x[i], 0.75f, -mx);
#pragma unroll
    for (int i = 0; i < 64; ++i)
        x[i] = __builtin_amdgcn_exp2f(x[i]);
    float l0 = 0.f, l1 = 0.f, l2 = 0.f, l3 = 0.f;
#pragma unroll
    for (int i = 0; i < 64; i += 4) {
        l0 += x[i];
        l1 += x[i + 1];
        l2 += x[i + 2];
        l3 += x[i + 3];
    }
    l = l * alpha + ((l0 + l1) + (l2 + l3));
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        s16x2 w = __builtin_bit_cast(s16x2, pk[i]);
        w = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(w, x[4 * i], x[4 * i + 1], 0.00390625f, false);
        w = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(w, x[4 * i + 2], x[4 * i + 3], 0.00390625f, true);
        pk[i] = __builtin_bit_cast(uint32_t, w);
    }
    coexec_rescale(ov, alpha);
}

// One stream per wave (kind 0: matrix, 1: vector) for `iters` iterations;
// returns a checksum of the stream's final state and the s_memtime cycles.
template <int KIND, int PAT>
__device__ float coexec_run(int iters, int lane, unsigned long long& cyc)
{
    unsigned long long t0, t1;
    float sum = 0.f;
    if constexpr (KIND == 0) {
        f32x16 acc[4], o[4];
        f32x4 q[4];
        for (int i = 0; i < 4; ++i)
            for (int r = 0; r < 16; ++r) {
                acc[i][r] = 0.f;
                o[i][r] = 0.f;
                q[i][r & 3] = 0.f;
            }
        bf16x8 a, b;
        i32x8 a8, b8;
        for (int i = 0; i < 8; ++i) {
            a[i] = (__bf16)(0.0078125f * (float)((lane + i) & 7));
            b[i] = (__bf16)(0.0078125f * (float)(i + 1));
            a8[i] = 0x30303030;     // E4M3 0.5 in every byte
            b8[i] = 0x20202020;     // E4M3 0.0625
        }
        asm volatile("s_memtime %0\n\ts_waitcnt lgkmcnt(0)" : "=s"(t0) :: "memory");
        for (int it = 0; it < iters; ++it)
            coexec_mfma<PAT>(acc, o, q, a, b, a8, b8);
        asm volatile("s_memtime %0\n\ts_waitcnt lgkmcnt(0)" : "=s"(t1) :: "memory");
        for (int i = 0; i < 4; ++i)
            for (int r = 0; r < 16; ++r)
                sum += acc[i][r] + o[i][r] + q[i][r & 3];
    } else {
        float x[64], ov[64];
        uint32_t pk[16];
        for (int i = 0; i < 64; ++i) {
            x[i] = -0.015625f * (float)((i + lane) & 31);
            ov[i] = 1.f;
        }
        for (int i = 0; i < 16; ++i)
            pk[i] = 0;
        float l = 0.f, mc = 0.f;
        asm volatile("s_memtime %0\n\ts_waitcnt lgkmcnt(0)" : "=s"(t0) :: "memory");
        for (int it = 0; it < iters; ++it)
            coexec_valu(x, ov, pk, l, mc);
        asm volatile("s_memtime %0\n\ts_waitcnt lgkmcnt(0)" : "=s"(t1) :: "memory");
        sum = l;
        for (int i = 0; i < 64; ++i)
            sum += x[i] + ov[i];
        for (int i = 0; i < 16; ++i)
            sum += (float)(pk[i] & 0xFFu);
    }
    cyc = t1 - t0;
    return sum;
}

// layout 0: waves 0-3 (one per SIMD) run the matrix stream; layout 1: waves 0-3
// run the vector stream; layout 2: 8 waves, wave w and wave w + 4 share SIMD
// w, waves 0-3 run the matrix stream and waves 4-7 the vector stream.
// The matrix stream is pattern PAT.  cycles[wg * 8 + wave] gets the wave's
// cycles, sink[wg * 512 + thread] its checksum.
template <int PAT>
__global__ void __launch_bounds__(512) k_coexec(int iters, int layout, unsigned long long* cycles, float* sink)
{
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int kind = layout == 2 ? (w < 4 ? 0 : 1) : layout;
    unsigned long long cyc = 0;
    const float sum = kind == 0 ? coexec_run<0, PAT>(iters, lane, cyc) : coexec_run<1, 0>(iters, lane, cyc);
    sink[blockIdx.x * 512 + threadIdx.x] = sum;
    if (lane == 0)
        cycles[blockIdx.x * 8 + w] = cyc;
}

// layout 3: waves 0-3, one per SIMD with the whole register file, each run both
// streams per iteration (the compiler interleaves them); the vector stream's
// multiplies rescale the P.V accumulators, as in the attention kernels
__global__ void __launch_bounds__(512) k_coexec_one(int iters, unsigned long long* cycles, float* sink)
{
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    f32x16 acc[4], o[4];
    for (int i = 0; i < 4; ++i)
        for (int r = 0; r < 16; ++r) {
            acc[i][r] = 0.f;
            o[i][r] = 0.f;
        }
    bf16x8 a, b;
    i32x8 a8, b8;
    for (int i = 0; i < 8; ++i) {
        a[i] = (__bf16)(0.0078125f * (float)((lane + i) & 7));
        b[i] = (__bf16)(0.0078125f * (float)(i + 1));
        a8[i] = 0x30303030;
        b8[i] = 0x20202020;
    }
    float x[64];
    uint32_t pk[16];
    for (int i = 0; i < 64; ++i)
        x[i] = -0.015625f * (float)((i + lane) & 31);
    for (int i = 0; i < 16; ++i)
        pk[i] = 0;
    float l = 0.f, mc = 0.f;
    unsigned long long t0, t1;
    asm volatile("s_memtime %0\n\ts_waitcnt lgkmcnt(0)" : "=s"(t0) :: "memory");
    f32x4 q[4] = {};
    for (int it = 0; it < iters; ++it) {
        coexec_mfma<0>(acc, o, q, a, b, a8, b8);
        coexec_valu(x, o, pk, l, mc);
    }
    asm volatile("s_memtime %0\n\ts_waitcnt lgkmcnt(0)" : "=s"(t1) :: "memory");
    float sum = l;
    for (int i = 0; i < 4; ++i)
        for (int r = 0; r < 16; ++r)
            sum += acc[i][r] + o[i][r];
    for (int i = 0; i < 64; ++i)
        sum += x[i];
    for (int i = 0; i < 16; ++i)
        sum += (float)(pk[i] & 0xFFu);
    sink[blockIdx.x * 512 + threadIdx.x] = sum;
    if (lane == 0)
        cycles[blockIdx.x * 8 + w] = t1 - t0;
}

extern "C" {

int probe_cvt_range(uint32_t lo, int64_t n, uint8_t* out, void* stream)
{
    if (n <= 0 || !out || (uint64_t)lo + (uint64_t)n > 0x100000000ull)
        return -1;
    hipLaunchKernelGGL(k_cvt_range, dim3(grid_for((n + 1) / 2, 256)), dim3(256), 0,
                       (hipStream_t)stream, lo, n, out);
    return hipGetLastError() == hipSuccess ? 0 : -3;
}

int probe_cvt_list(const float* x, int64_t n, uint8_t* out, float scale, int scaled, int hi,
                   void* stream)
{
    if (n <= 0 || !x || !out)
        return -1;
    hipLaunchKernelGGL(k_cvt_list, dim3(grid_for((n + 1) / 2, 256)), dim3(256), 0,
                       (hipStream_t)stream, x, n, out, scale, scaled, hi);
    return hipGetLastError() == hipSuccess ? 0 : -3;
}

int probe_exp2(const float* x, int64_t n, float* out, void* stream)
{
    if (n <= 0 || !x || !out)
        return -1;
    hipLaunchKernelGGL(k_exp2, dim3(grid_for(n, 256)), dim3(256), 0, (hipStream_t)stream, x, n, out);
    return hipGetLastError() == hipSuccess ? 0 : -3;
}

int probe_mfma_fp8_scaled(const uint8_t* A, const uint8_t* B, const uint8_t* sa, const uint8_t* sb,
                          float* D, void* stream)
{
    if (!A || !B || !sa || !sb || !D)
        return -1;
    hipLaunchKernelGGL(k_mfma_fp8_scaled, dim3(1), dim3(64), 0, (hipStream_t)stream, A, B, sa, sb, D);
    return hipGetLastError() == hipSuccess ? 0 : -3;
}

// n must be even (pairs)
int probe_cvt_scaled_vec(const float* x, const float* scale, int64_t n, uint8_t* out, void* stream)
{
    if (n <= 0 || (n & 1) || !x || !scale || !out)
        return -1;
    hipLaunchKernelGGL(k_cvt_scaled_vec, dim3(grid_for(n / 2, 256)), dim3(256), 0, (hipStream_t)stream,
                       x, scale, n, out);
    return hipGetLastError() == hipSuccess ? 0 : -3;
}

// `out` holds blocks * 256 floats; exp2 evaluations = blocks * 256 * iters * 16
int probe_exp2_rate(int blocks, int iters, float* out, void* stream)
{
    if (blocks <= 0 || iters <= 0 || !out)
        return -1;
    hipLaunchKernelGGL(k_exp2_rate, dim3(blocks), dim3(256), 0, (hipStream_t)stream, iters, out);
    return hipGetLastError() == hipSuccess ? 0 : -3;
}

int probe_lds_rate(int blocks, int iters, int mode, int readers, int copiers, const void* src,
                   unsigned long long* cycles, uint32_t* sink, void* stream)
{
    if (blocks <= 0 || iters <= 0 || mode < 0 || mode > 1 || readers < 0 || copiers < 0 ||
        readers + copiers > 8 || !cycles || !sink || (copiers > 0 && !src))
        return -1;
    hipLaunchKernelGGL(k_lds_rate, dim3(blocks), dim3(512), 0, (hipStream_t)stream, iters, mode, readers,
                       copiers, (const uint8_t*)src, cycles, sink);
    return hipGetLastError() == hipSuccess ? 0 : -3;
}

int probe_mfma(int which, const void* A, const void* B, float* D, void* stream)
{
    if (!A || !B || !D)
        return -1;
    hipStream_t s = (hipStream_t)stream;
    if (which == 0)
        hipLaunchKernelGGL(k_mfma_bf16, dim3(1), dim3(64), 0, s, (const uint16_t*)A, (const uint16_t*)B, D);
    else if (which == 1)
        hipLaunchKernelGGL(k_mfma_fp8, dim3(1), dim3(64), 0, s, (const uint8_t*)A, (const uint8_t*)B, D);
    else if (which == 2)
        hipLaunchKernelGGL(k_mfma_f32, dim3(1), dim3(64), 0, s, (const float*)A, (const float*)B, D);
    else
        return -1;
    return hipGetLastError() == hipSuccess ? 0 : -3;
}

// cycles: blocks * 8 entries, sink: blocks * 512 floats (layouts 0, 1 and 3
// write waves 0-3 only); pattern: the matrix stream of layouts 0 and 2 (0-3;
// layout 3 runs pattern 0)
int probe_coexec(int blocks, int iters, int layout, int pattern, unsigned long long* cycles, float* sink,
                 void* stream)
{
    if (blocks <= 0 || iters <= 0 || layout < 0 || layout > 3 || pattern < 0 || pattern > 3 || !cycles || !sink)
        return -1;
    hipStream_t s = (hipStream_t)stream;
    const dim3 blk(layout == 2 ? 512 : 256);
    if (layout == 3)
        hipLaunchKernelGGL(k_coexec_one, dim3(blocks), dim3(256), 0, s, iters, cycles, sink);
    else if (pattern == 0)
        hipLaunchKernelGGL(k_coexec<0>, dim3(blocks), blk, 0, s, iters, layout, cycles, sink);
    else if (pattern == 1)
        hipLaunchKernelGGL(k_coexec<1>, dim3(blocks), blk, 0, s, iters, layout, cycles, sink);
    else if (pattern == 2)
        hipLaunchKernelGGL(k_coexec<2>, dim3(blocks), blk, 0, s, iters, layout, cycles, sink);
    else
        hipLaunchKernelGGL(k_coexec<3>, dim3(blocks), blk, 0, s, iters, layout, cycles, sink);
    return hipGetLastError() == hipSuccess ? 0 : -3;
}

}  // extern "C"
