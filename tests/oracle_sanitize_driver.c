/*
 * Driver for the oracle under AddressSanitizer and UndefinedBehaviorSanitizer
 * (host code only; built and run by tests/test_oracle_sanitize.py with gcc).
 * It links oracle/oracle.c directly and calls its entry points over small
 * seeded inputs covering every option: both orders, causal and not, cast on
 * and off, static and dynamic scales, descales, the code-ambiguity bound, the
 * per-block diagnostic, row subsets, several threads, and queries against a
 * longer KV cache.  Besides the sanitizers' own checks it asserts a few
 * properties that hold for any input:
 *   - every E4M3 code decodes and re-encodes to itself, NaN up to its sign
 *     (Sec. 2.1);
 *   - the encoder is monotone over a sweep of FP32 bit patterns;
 *   - a row subset gives bit-identical rows to the full run;
 *   - with the cast off, S = 2^k gives bit-identical outputs to S = 1
 *     (Prop. 2: scaling by a power of two commutes with every rounding).
 * Exit status 0 when all hold.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

uint8_t oracle_e4m3_encode(float y);
float oracle_e4m3_decode(uint8_t code);
int oracle_attn_full(const float* q, const float* k, const float* v, float* out, float* lse,
                     uint32_t* counts, float* amb, uint32_t* gap_hist, uint32_t* blk_zero,
                     int nbins, int B, int Hq, int Hkv, int Nq, int Nk, int d, int causal,
                     int block_kv, int order, float S, int cast, int scale_mode, int n_sink,
                     float q_descale, float k_descale, float v_descale, double amb_rel,
                     double jitter_rel, const int64_t* rows, int64_t n_rows, int nthreads);
int oracle_ref_fp64_kv(const float* q, const float* k, const float* v, double* out,
                       double* lse, int B, int Hq, int Hkv, int Nq, int Nk, int d, int causal,
                       double q_descale, double k_descale, double v_descale,
                       const int64_t* rows, int64_t n_rows, int nthreads);

static int failures = 0;
#define CHECK(cond, ...)                                                    \
    do {                                                                    \
        if (!(cond)) {                                                      \
            fprintf(stderr, "FAIL %s:%d: ", __FILE__, __LINE__);            \
            fprintf(stderr, __VA_ARGS__);                                   \
            fputc('\n', stderr);                                            \
            failures++;                                                     \
        }                                                                   \
    } while (0)

/* xorshift64*: seeded uniform numbers for the inputs */
static uint64_t rng_state = 0x243F6A8885A308D3ull;
static double urand(void)
{
    rng_state ^= rng_state >> 12;
    rng_state ^= rng_state << 25;
    rng_state ^= rng_state >> 27;
    return (double)((rng_state * 0x2545F4914F6CDD1Dull) >> 11) * 0x1p-53;
}

/* values on the 2^-5 grid in [-4, 4): every dot product is exact */
static float grid_value(void) { return (float)(floor(urand() * 256.0) - 128.0) / 32.0f; }

static float* alloc_fill(size_t n, int grid)
{
    float* a = (float*)malloc(n * sizeof(float));
    for (size_t i = 0; i < n; i++)
        a[i] = grid ? grid_value() : (float)(urand() * 2.0 - 1.0);
    return a;
}

static void codec_checks(void)
{
    for (int c = 0; c < 256; c++) {
        const float v = oracle_e4m3_decode((uint8_t)c);
        const uint8_t back = oracle_e4m3_encode(v);
        if ((c & 0x7F) == 0x7F) {          /* NaN: the code, up to its sign bit */
            CHECK((back & 0x7F) == 0x7F, "NaN code 0x%02x re-encodes to 0x%02x", c, back);
            continue;
        }
        CHECK(back == (uint8_t)c, "code 0x%02x decodes to %g, re-encodes to 0x%02x", c, v, back);
    }
    /* monotone over positive finite FP32 patterns (every 65537th) */
    uint8_t prev = 0;
    for (uint64_t u = 0; u < 0x7F800000ull; u += 65537) {
        float y;
        const uint32_t b = (uint32_t)u;
        memcpy(&y, &b, 4);
        const uint8_t e = oracle_e4m3_encode(y);
        CHECK(e >= prev, "encode not monotone at 0x%08x", b);
        prev = e;
    }
}

static void attn_checks(int B, int Hq, int Hkv, int Nq, int Nk, int d, int bc)
{
    const size_t nq = (size_t)B * Hq * Nq * d, nk = (size_t)B * Hkv * Nk * d;
    float* q = alloc_fill(nq, 1);
    float* k = alloc_fill(nk, 1);
    float* v = alloc_fill(nk, 0);
    const int64_t rows = (int64_t)B * Hq * Nq;
    const int nblk = (Nk + bc - 1) / bc;
    float* out = (float*)malloc((size_t)rows * d * sizeof(float));
    float* out2 = (float*)malloc((size_t)rows * d * sizeof(float));
    float* amb = (float*)malloc((size_t)rows * d * sizeof(float));
    float* lse = (float*)malloc((size_t)rows * sizeof(float));
    uint32_t* cnt = (uint32_t*)malloc((size_t)rows * 3 * sizeof(uint32_t));
    uint32_t* hist = (uint32_t*)malloc((size_t)B * Hq * nblk * 16 * sizeof(uint32_t));
    uint32_t* bz = (uint32_t*)malloc((size_t)B * Hq * nblk * sizeof(uint32_t));
    double* ref = (double*)malloc((size_t)rows * d * sizeof(double));
    double* rlse = (double*)malloc((size_t)rows * sizeof(double));
    int64_t* sub = (int64_t*)malloc((size_t)rows * sizeof(int64_t));
    int64_t n_sub = 0;
    for (int64_t r = rows - 1; r >= 0; r -= 3)
        sub[n_sub++] = r;                               /* descending subset */
    float* out_s = (float*)malloc((size_t)n_sub * d * sizeof(float));
    uint32_t* cnt_s = (uint32_t*)malloc((size_t)n_sub * 3 * sizeof(uint32_t));

    for (int causal = 0; causal < 2; causal++)
        for (int order = 0; order < 2; order++)
            for (int dyn = 0; dyn < 2; dyn++) {
                const float S = dyn ? 16.0f : 256.0f;
                int rc = oracle_attn_full(q, k, v, out, lse, cnt, amb, hist, bz, 16, B, Hq, Hkv,
                                          Nq, Nk, d, causal, bc, order, S, 1, dyn, 4, 0.75f, 1.5f,
                                          2.0f, 6.0 * 0x1p-23, 0.0, NULL, rows, 3);
                CHECK(rc == 0, "oracle_attn_full rc %d", rc);
                rc = oracle_attn_full(q, k, v, out_s, NULL, cnt_s, NULL, NULL, NULL, 0, B, Hq,
                                      Hkv, Nq, Nk, d, causal, bc, order, S, 1, dyn, 4, 0.75f,
                                      1.5f, 2.0f, 0.0, 0.0, sub, n_sub, 2);
                CHECK(rc == 0, "subset rc %d", rc);
                for (int64_t i = 0; i < n_sub; i++) {
                    CHECK(memcmp(out_s + i * d, out + sub[i] * d, (size_t)d * 4) == 0,
                          "subset row %lld differs", (long long)sub[i]);
                    CHECK(memcmp(cnt_s + 3 * i, cnt + 3 * sub[i], 12) == 0,
                          "subset counts of row %lld differ", (long long)sub[i]);
                }
                /* cast off: S = 2^k bit-identical to S = 1 */
                rc = oracle_attn_full(q, k, v, out, NULL, NULL, NULL, NULL, NULL, 0, B, Hq, Hkv,
                                      Nq, Nk, d, causal, bc, order, 1.0f, 0, 0, 4, 1.0f, 1.0f,
                                      1.0f, 0.0, 0.0, NULL, rows, 4);
                CHECK(rc == 0, "cast-off rc %d", rc);
                rc = oracle_attn_full(q, k, v, out2, NULL, NULL, NULL, NULL, NULL, 0, B, Hq, Hkv,
                                      Nq, Nk, d, causal, bc, order, 256.0f, 0, 0, 4, 1.0f, 1.0f,
                                      1.0f, 0.0, 0.0, NULL, rows, 4);
                CHECK(rc == 0, "cast-off rc %d", rc);
                CHECK(memcmp(out, out2, (size_t)rows * d * 4) == 0,
                      "cast off: S = 256 differs from S = 1 (causal %d order %d)", causal, order);
                rc = oracle_ref_fp64_kv(q, k, v, ref, rlse, B, Hq, Hkv, Nq, Nk, d, causal, 0.75,
                                        1.5, 2.0, NULL, rows, 3);
                CHECK(rc == 0, "ref rc %d", rc);
            }
    /* invalid arguments are rejected, not read */
    CHECK(oracle_attn_full(q, k, v, out, lse, cnt, NULL, NULL, NULL, 0, B, Hq, Hkv, Nq, Nk, d, 0,
                           bc, 0, 256.0f, 1, 0, 4, 1.0f, 1.0f, 1.0f, 0.0, 0.01, NULL, rows, 1)
              == -1, "planted error accepted outside the test build");
    CHECK(oracle_attn_full(q, k, v, out, lse, cnt, NULL, NULL, NULL, 0, B, Hq, Hkv, Nq, Nk, d, 0,
                           bc, 0, 3.0f, 1, 1, 4, 1.0f, 1.0f, 1.0f, 0.0, 0.0, NULL, rows, 1) == -1,
          "dynamic scale with S = 3 accepted");
    free(q); free(k); free(v); free(out); free(out2); free(amb); free(lse); free(cnt);
    free(hist); free(bz); free(ref); free(rlse); free(sub); free(out_s); free(cnt_s);
}

int main(void)
{
    codec_checks();
    attn_checks(2, 4, 2, 133, 133, 64, 64);      /* square, ragged last block, GQA */
    attn_checks(1, 2, 1, 37, 300, 128, 128);     /* queries against a longer cache */
    attn_checks(1, 1, 1, 1, 1, 64, 64);          /* one row, one key */
    if (failures) {
        fprintf(stderr, "%d check(s) failed\n", failures);
        return 1;
    }
    printf("oracle sanitizer driver: all checks passed\n");
    return 0;
}
