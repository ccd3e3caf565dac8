/*
 * attn_fp8.h -- C ABI of libattn_fp8.so: FP8 online-softmax attention forward
 * for AMD Instinct MI355X (gfx950), with a static P-scale S and a runtime
 * KV-block iteration order.
 *
 * The operation is the FP8 online-softmax attention of Algorithm 1 in
 * "P-Cast Precision in FP8 Attention: Sink-Induced Collapse and the Optimality
 * of S = 2^8" (Sec. 2.2), applied to every query row of every (batch, head),
 * with the kernel semantics of Sec. 6.1.  Each row keeps a running maximum of
 * its scores, a running sum l and an FP32 output accumulator, and visits its
 * KV blocks one at a time in the chosen order.  Per block, the maximum is
 * raised to cover the block's scores and the old l and accumulator are
 * rescaled to it; l then adds the block's softmax numerators P in FP32
 * before any cast (the normaliser is exact), while the accumulator adds
 * products of V with the E4M3 codes of P * S (round to nearest even), so the
 * cast error sits in the numerator alone.  The result is the accumulator
 * divided by S * l.
 * The device works in base 2: with c = fl32(log2(e)/sqrt(d)) and D the raw
 * dot product q.k, mc = fl(m*c), x = fma(D, c, -mc), P = exp2(x), and the
 * rescale factor is exp2(mc_old - mc_new).  KV blocks are [j*block_kv,
 * (j+1)*block_kv) anchored at key 0; ATTN_ORDER_FORWARD visits j = 0, 1, ...;
 * ATTN_ORDER_REVERSE visits the last block first and the sink block (block 0)
 * last (Sec. 4.1).  Under causal masking, row r sees keys t <= r only and
 * visits only the blocks that hold at least one such key; masked keys take
 * no part in l, the accumulator or the counts.  The running maximum is
 * updated once per KV block, never lazily.
 *
 * Memory layout (all contiguous, row-major, device memory owned by the caller):
 *   q    [B][Hq][N][d]
 *   k, v [B][Hkv][N][d]      (query head h reads KV head h / (Hq/Hkv))
 *   out  [B][Hq][N][d]  float32
 *   lse  [B][Hq][N]     float32, natural-log log-sum-exp of z = q.k/sqrt(d)
 *                               over the row's valid keys (independent of S)
 *   counts [B][Hq][N][3] uint32 (p_underflow_count only)
 *
 * Element types by mode:
 *   ATTN_MODE_FAITHFUL : q, k, v float32.  Scores and P.V on FP32 MFMA; exp2
 *                        evaluated in FP64 and rounded to FP32; P*S rounded to
 *                        E4M3 by the hardware convert and decoded back to FP32
 *                        (Sec. 6.1: Q, K, V kept in FP32 to isolate the cast).
 *   ATTN_MODE_FAST     : q, k bfloat16 (raw 16-bit patterns), v OCP E4M3 bytes.
 *                        Scores on the bf16 MFMA, exp2 by the hardware
 *                        instruction, E4M3 P bytes straight into the FP8 MFMA.
 *   ATTN_MODE_NOCAST   : like FAITHFUL with the cast disabled (P*S used as is);
 *                        a diagnostic for the FP64 comparison.
 *   ATTN_MODE_FP8QK    : q, k and v all OCP E4M3 bytes.  Scores on the FP8 MFMA,
 *                        the FP8 x FP8 -> FP32 scores of Algorithm 1; otherwise
 *                        as FAST.  Per-tensor descales (Sec. 6.1: QKV
 *                        quantization carries its own qscale/kscale/vscale) go
 *                        through the *_descaled entry points.
 *   The E4M3 cast saturates: P*S >= 448 becomes 448 (reachable only for S > 448).
 *
 * Alignment: q, k, v and out must be 16-byte aligned (the kernels move them in
 * 16-byte vectors; rows of a contiguous tensor then stay aligned because
 * d is 64 or 128), lse, counts and the diagnostic arrays 4-byte aligned;
 * otherwise ATTN_ERR_INVALID_ARG.
 *
 * Ownership and threading: every pointer is a device pointer owned by the
 * caller.  The library allocates no memory and keeps no state between calls;
 * it is reentrant.  The one scratch buffer a call can use, the workspace of a
 * KV-cache call whose 32-row tiles cannot fill the GPU (see attn_fp8_fwd_kv),
 * is passed in by the caller.  Work is enqueued on `stream` (a hipStream_t;
 * NULL = the null stream) and runs asynchronously: a return of ATTN_OK means
 * "validated and launched"; synchronise on the stream before reading results.
 *
 * Errors: arguments are validated before any HIP call; on failure nothing is
 * launched and the return value says why.  A launch failure reported by the
 * HIP runtime returns ATTN_ERR_HIP.  No C++ exception crosses this interface.
 */
#ifndef ATTN_FP8_H
#define ATTN_FP8_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    ATTN_MODE_FAITHFUL = 0,
    ATTN_MODE_FAST = 1,
    ATTN_MODE_NOCAST = 2,
    ATTN_MODE_FP8QK = 3
};

/*
 * Flag OR-ed into `mode`: dynamic per-block power-of-two P-scale (the
 * paper's Limitations and Future Work proposes scaling each block by a power
 * of two chosen from its own P range, without fixing the rule).  Rule used
 * here: S must be 2^k0 with 0 <= k0 <= 8; block j of query row r casts
 * P * 2^kj with
 *   kj = k0 + clamp(floor(-xmax), 0, 126 - k0),  xmax = fma(mloc, c, -mc),
 * mloc the block's largest raw score of the row and mc = fl(m_new c), so the
 * block's largest P lands in (S/2, S] like P = 1 does under the static S; a
 * block holding the running maximum keeps kj = k0.  The cast value is taken
 * back to S units exactly (times 2^(k0 - kj)), so l, O and the epilogue are
 * those of the static scale.  With ATTN_MODE_NOCAST the flag changes nothing.
 */
enum { ATTN_SCALE_DYNAMIC = 0x100 };

/*
 * Flags OR-ed into `mode` (fast modes, self-attention and long query chunks
 * of a KV cache): the schedule of the persistent kernel.
 *   ATTN_TILE_256  256 query rows per tile, eight waves of 32 rows, every
 *                  wave over every KV block of its rows; tiles t and T-1-t of
 *                  a head form one work unit (equal causal work per unit).
 *   ATTN_TILE_128  128 query rows per tile, one tile per work unit; the two
 *                  waves of a 32-row group take alternate KV blocks of the
 *                  visit and hand the running maximum to each other, so every
 *                  block still sees the running maximum of Algorithm 1.
 * Neither: ATTN_TILE_256, unless its units leave compute units idle and a
 * cost model of the two schedules' critical paths favours ATTN_TILE_128.
 * Both: ATTN_ERR_INVALID_ARG.  The two schedules
 * give identical E4M3 codes and counts; O and l differ only in FP32 rounding
 * (each 128-row group adds two partial sums at the end).  No effect in the
 * other modes or on short query chunks.
 */
enum { ATTN_TILE_256 = 0x200, ATTN_TILE_128 = 0x400 };

enum {
    ATTN_ORDER_FORWARD = 0, /* KV blocks 0, 1, ..., last (sink block first)  */
    ATTN_ORDER_REVERSE = 1  /* KV blocks last, ..., 1, 0 (sink block last)   */
};

enum {
    ATTN_OK = 0,
    ATTN_ERR_INVALID_ARG = -1, /* null pointer, bad shape, S not finite/positive, ... */
    ATTN_ERR_UNSUPPORTED = -2, /* valid but not built: d or block_kv outside {64,128},
                                  more than 2^30 keys per (batch, head) */
    ATTN_ERR_HIP = -3,         /* the HIP runtime rejected the launch */
    ATTN_ERR_SCRATCH = -4      /* attn_fp8_fwd_kv_noalloc: shape needs more than its scratch */
};

/*
 * Attention forward (Algorithm 1 over every row).
 *   q, k, v   device inputs, element type by `mode` (see above).
 *   out       device float32 [B][Hq][N][d]; required.
 *   lse       device float32 [B][Hq][N]; may be NULL.
 *   B, Hq, Hkv, N, d
 *             batch, query heads, KV heads (Hq % Hkv == 0), sequence length,
 *             head dimension (64 or 128).  N may be any value in [0, 2^30]
 *             (beyond: ATTN_ERR_UNSUPPORTED); B*Hq*N == 0 is a no-op
 *             (pointers are then not inspected).
 *   causal    0 or 1.
 *   block_kv  KV block size B of Algorithm 1: 64 or 128.  It is the granularity
 *             of the running-maximum update and therefore part of the result.
 *   order     ATTN_ORDER_FORWARD or ATTN_ORDER_REVERSE.
 *   S         static P-scale (Sec. 5), finite and > 0.  Powers of two make the
 *             scaling exact (Prop. 2); S = 256 is the paper's choice.
 *   mode      ATTN_MODE_*, optionally OR ATTN_SCALE_DYNAMIC and one ATTN_TILE_*.
 *   stream    hipStream_t or NULL.
 * Returns ATTN_OK or an ATTN_ERR_* code.
 */
int attn_fp8_fwd(const void* q, const void* k, const void* v, float* out,
                 float* lse, int B, int Hq, int Hkv, int N, int d, int causal,
                 int block_kv, int order, float S, int mode, void* stream);

/*
 * P-underflow diagnostic (Prop. 1): runs the same computation as attn_fp8_fwd
 * and, for every query row, counts the valid keys whose cast code
 * E4M3(P*S) is zero, split by key position:
 *   counts[row][0]: keys t <  n_sink                 (the sink keys)
 *   counts[row][1]: keys n_sink <= t < block_kv      (non-sink keys sharing
 *                                                     the sink's KV block)
 *   counts[row][2]: keys t >= block_kv               (all other blocks)
 *   counts    device uint32 [B][Hq][N][3]; required; every entry is written.
 *   n_sink    0 <= n_sink <= block_kv (the sink keys lie in block 0, so the
 *             three categories are disjoint); else ATTN_ERR_INVALID_ARG.
 *   out, lse  optional (NULL allowed); when given they receive the same
 *             values attn_fp8_fwd writes.
 * Other arguments and return codes as for attn_fp8_fwd.
 */
int attn_fp8_p_underflow_count(const void* q, const void* k, const void* v,
                               int B, int Hq, int Hkv, int N, int d, int causal,
                               int block_kv, int order, float S, int mode,
                               int n_sink, uint32_t* counts, float* out,
                               float* lse, void* stream);

/*
 * The two entry points above with per-tensor descales: the stored q, k, v
 * values stand for q*q_descale, k*k_descale, v*v_descale (Sec. 6.1: the QKV
 * quantization has its own scales, separate from the P-scale S).  With D the
 * raw dot product of the stored q and k, the scores are
 * z = D q_descale k_descale / sqrt(d): the device uses
 * c = fl32(log2(e) q_descale k_descale / sqrt(d)) (rounded once from double)
 * in place of log2(e)/sqrt(d), and the output is O / (S l) times v_descale.
 * The plain entry points are these with all three descales 1.  Descales must
 * be finite and > 0, else ATTN_ERR_INVALID_ARG.
 */
int attn_fp8_fwd_descaled(const void* q, const void* k, const void* v, float* out,
                          float* lse, int B, int Hq, int Hkv, int N, int d,
                          int causal, int block_kv, int order, float S, int mode,
                          float q_descale, float k_descale, float v_descale,
                          void* stream);

int attn_fp8_p_underflow_count_descaled(const void* q, const void* k, const void* v,
                                        int B, int Hq, int Hkv, int N, int d,
                                        int causal, int block_kv, int order, float S,
                                        int mode, int n_sink, float q_descale,
                                        float k_descale, float v_descale,
                                        uint32_t* counts, float* out, float* lse,
                                        void* stream);

/*
 * Queries against a KV cache: Nq query rows per (batch, head) against Nk
 * cached keys (0 <= Nq <= Nk), the prefill shape of the paper's Exp. 1
 * (q_len = 32 against N = 4096) and of the prefill kernel it simulates
 * (Sec. 6: kernel-faithful simulation).  Query row r is the token at key position
 * Nk - Nq + r (the queries are the last Nq positions); with causal = 1 it
 * sees keys 0 .. Nk - Nq + r, otherwise all Nk.  Algorithm 1 is unchanged:
 * every row visits its KV blocks [j*block_kv, (j+1)*block_kv) in the given
 * order, the P-cast and the counts follow the row's sequential running
 * maximum exactly.
 *
 *   q    [B][Hq][Nq][d], k and v [B][Hkv][Nk][d] (dtypes as for the mode);
 *   out  [B][Hq][Nq][d] float32, lse [B][Hq][Nq] (optional),
 *   counts [B][Hq][Nq][3] (count variant).
 *
 * With Nq = Nk these are attn_fp8_fwd_descaled / _p_underflow_count_descaled.
 * With Nq < Nk the fast modes run on a prefill kernel: the eight waves of a
 * workgroup split a 32-row tile's KV blocks into contiguous ranges of the
 * visit order; each range starts from the running maximum the row reached
 * before it, so the P codes are those of the sequential visit; only the FP32
 * summation order of O and l differs.  (Long chunks, Nq >= 128 with Nk - Nq a
 * multiple of block_kv, run on the square problem's kernel instead.)  When
 * the tiles are fewer than the GPU's compute units, each tile can be split
 * over C = min(CUs / tiles, blocks / 8, 8) workgroups; the call then enqueues
 * three kernels (the range maxima, Algorithm 1 per range, a merge) and needs
 * a device workspace of attn_fp8_kv_workspace_bytes() bytes:
 *   workspace        device memory of the caller, 256-byte aligned, or NULL.
 *                    The call uses it as scratch on `stream` (no contents are
 *                    read before the call writes them); calls that overlap in
 *                    time must not share one.  NULL runs the tiles unsplit
 *                    (same results, fewer workgroups).
 *   workspace_bytes  its size; with a non-NULL workspace it must be at least
 *                    what attn_fp8_kv_workspace_bytes reports for the same
 *                    shape on the current device, else ATTN_ERR_INVALID_ARG.
 * Nq > Nk returns ATTN_ERR_INVALID_ARG, Nk > 2^30 ATTN_ERR_UNSUPPORTED; other
 * arguments and return codes as
 * for the descaled entry points.
 */
int attn_fp8_fwd_kv(const void* q, const void* k, const void* v, float* out, float* lse,
                    int B, int Hq, int Hkv, int Nq, int Nk, int d, int causal,
                    int block_kv, int order, float S, int mode, float q_descale,
                    float k_descale, float v_descale, void* workspace,
                    size_t workspace_bytes, void* stream);

int attn_fp8_p_underflow_count_kv(const void* q, const void* k, const void* v, int B,
                                  int Hq, int Hkv, int Nq, int Nk, int d, int causal,
                                  int block_kv, int order, float S, int mode, int n_sink,
                                  float q_descale, float k_descale, float v_descale,
                                  uint32_t* counts, float* out, float* lse,
                                  void* workspace, size_t workspace_bytes, void* stream);

/*
 * attn_fp8_fwd_kv without a workspace argument and without allocating: for
 * callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc).  The KV-cache split
 * takes its scratch from a fixed device array inside the library instead:
 * 8 MiB per GPU, created when the library's code is loaded on that GPU and
 * held until the process ends.  The split never needs more than
 * CUs * (32 d + 288) * 4 + 512 bytes (4.5 MB on a 256-CU MI355X at d = 128);
 * a shape that would returns ATTN_ERR_SCRATCH, with nothing launched.  Every
 * call on one GPU shares that GPU's array: calls that overlap in time on one
 * GPU (different streams or host threads) race and must be serialised by the
 * caller.  No call reads scratch contents it did not write itself.  Arguments,
 * results and other return codes as for attn_fp8_fwd_kv.
 */
int attn_fp8_fwd_kv_noalloc(const void* q, const void* k, const void* v, float* out,
                            float* lse, int B, int Hq, int Hkv, int Nq, int Nk, int d,
                            int causal, int block_kv, int order, float S, int mode,
                            float q_descale, float k_descale, float v_descale,
                            void* stream);

/*
 * Workspace the KV-cache entry points can use for the shape (B, Hq, Hkv, Nq,
 * Nk, d, causal, block_kv, mode) on the current device: *bytes is set to 0
 * when the call would not split (square problems, long chunks, faithful
 * modes, tiles enough to fill the GPU), else to the size of the range maxima
 * (tiles * C * 8 * 32 floats) plus, from a 256-byte boundary, the partial
 * sums (tiles * C * (32 d + 32) floats).  Since tiles * C never exceeds the
 * CU count, this stays below CUs * (32 d + 288) * 4 + 512 bytes (4.5 MB on a
 * 256-CU MI355X at d = 128).  Queries the device's CU count; launches nothing.
 * Returns ATTN_OK, ATTN_ERR_INVALID_ARG (bad shape, NULL bytes),
 * ATTN_ERR_UNSUPPORTED, or ATTN_ERR_HIP if the device cannot be queried.
 */
int attn_fp8_kv_workspace_bytes(int B, int Hq, int Hkv, int Nq, int Nk, int d, int causal,
                                int block_kv, int mode, size_t* bytes);

/*
 * Per-block diagnostic: where each KV block sits below the running maximum,
 * and how many of its P values the cast zeroes.  The paper's collapse
 * analysis assumes one sink cluster at key 0 and notes that with sinks spread
 * over the sequence the sink gap Delta is replaced by the gap of each block
 * (Limitations and Future Work, "Multi-sink patterns"; Prop. 1 for the
 * zero codes).  This call measures that gap per (row, block) on the device,
 * in the same pass as attn_fp8_p_underflow_count_descaled (same arguments,
 * same counts / out / lse), and adds two aggregates over the rows:
 *
 *   gap_hist  device uint32 [B][Hq][nblk][nbins], nblk = ceil(N / block_kv).
 *             For every row and every block j the row visits, with mx the
 *             block's largest raw score of the row, mc = fl(m_new c) and
 *             m_new the running maximum after block j, the gap
 *             g = -fma(mx, c, -mc) (log2 units: the block's largest P is
 *             2^-g) falls in bin min(max(floor(g), 0), nbins - 1), and
 *             gap_hist[b][h][j][bin] counts it.  A block holding the running
 *             maximum lands in bin 0; with S = 2^k the whole block is cast
 *             to zero exactly when g >= 10 + k.
 *   blk_zero  device uint32 [B][Hq][nblk]: zero codes of block j summed over
 *             the rows (valid keys only, same rule as counts).  Zero in
 *             no-cast mode.
 *   nbins     1 .. 64.
 *
 * Both arrays are cleared by the call on `stream` (by a kernel, no memset)
 * and filled with device atomics; their contents do not depend on the order
 * of those atomics.  Returns ATTN_ERR_INVALID_ARG if nbins is out of range or
 * a non-empty problem comes with a NULL gap_hist, blk_zero or counts; other
 * arguments and return codes as for attn_fp8_p_underflow_count_descaled.
 */
int attn_fp8_block_gap_diag(const void* q, const void* k, const void* v, int B, int Hq,
                            int Hkv, int N, int d, int causal, int block_kv, int order,
                            float S, int mode, int n_sink, float q_descale,
                            float k_descale, float v_descale, int nbins,
                            uint32_t* gap_hist, uint32_t* blk_zero, uint32_t* counts,
                            float* out, float* lse, void* stream);

/* Static, human-readable text for a status code (never NULL). */
const char* attn_fp8_strerror(int status);

/* Library version: major*10000 + minor*100 + patch. */
int attn_fp8_version(void);

#ifdef __cplusplus
}
#endif

#endif /* ATTN_FP8_H */
