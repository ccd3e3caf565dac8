/*
 * CPU oracle for FP8 online-softmax attention with a static P-scale S and a
 * runtime KV-block order.  TEST INFRASTRUCTURE ONLY: the product path never
 * links, loads or calls this file; tests, the smoke check and the benchmark's
 * CPU-baseline leg do.  It shares no code, header or table with the GPU
 * library.
 *
 * Plain, slow and sequential per query row.  Threads only split the list of
 * rows; every row is computed exactly as written below.
 *
 * What it follows in the paper:
 *   - E4M3 number line (Sec. 2.1, the subnormal and normal equations and the
 *     key-thresholds table): sign bit, 4 exponent bits with bias 7, 3 mantissa
 *     bits, subnormals M/8 * 2^-6, normals 2^(E-7) (1 + M/8), E=15,M=7 is NaN,
 *     max 448.
 *   - Algorithm 1 (FP8 online softmax attention, one query row) together with
 *     the kernel-faithful simulation rules of Sec. 6.1: l from the pre-cast
 *     FP32 P, O from the cast P, round-to-nearest E4M3 cast of P*S, epilogue
 *     O / (S * l).
 *   - Prop. 1 (P-underflow condition): a P value underflows when its code is
 *     zero; the diagnostic counts those codes per key category, and per
 *     block together with each block's gap below the running maximum
 *     (Limitations and Future Work, "Multi-sink patterns").
 *   - Limitations and Future Work, "worst-case vs average-case": a dynamic
 *     per-block power-of-two scale, chosen from the block's P range (only
 *     sketched in the paper; the rule below is this oracle's reading).
 *
 * Readings where the paper leaves the arithmetic open (each also listed in
 * the design notes of the repository):
 *   - scores use exp2 with c = log2(e)/sqrt(d) folded in, i.e.
 *     exp(z - m) = exp2(D*c - m*c) with D the raw dot q.k;
 *     mc = fl(m*c), x = fma(D, c, -mc), alpha = exp2(mc_old - mc_new);
 *   - exp2 is evaluated in double and rounded once to float;
 *   - the E4M3 cast is round-to-nearest-even, keeps subnormals, and saturates
 *     to +-448 (NaN stays NaN), so 2^-10 itself rounds to zero;
 *   - KV blocks are [j*Bc, (j+1)*Bc) anchored at key 0; reverse visits the
 *     last block first; under causal masking a row visits only the blocks
 *     holding at least one key t <= r, and masked keys take no part in l, O or
 *     the counts.
 *   - dynamic scale (scale_mode 1, S = 2^k0 with 0 <= k0 <= 8): block j of a
 *     row casts with S_j = 2^kj, kj = min(k0 + max(0, floor(-xmax)), 126),
 *     xmax = fma(max_t D_t, c, -mc) the block's largest exponent argument, so
 *     the block's largest P lands in (S/2, S] as the static scale puts P = 1;
 *     a block that holds the running maximum keeps kj = k0.  The decoded value
 *     is taken back to S units exactly (times 2^(k0 - kj)), so O, l and the
 *     epilogue are those of the static scale.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_VERSION 6

/* ------------------------------------------------------------------------- */
/* OCP E4M3 (Sec. 2.1)                                                        */
/* ------------------------------------------------------------------------- */

/* Decode one E4M3 byte: subnormal (E=0) v = M/8 * 2^-6, normal
 * v = 2^(E-7) * (1 + M/8); E=15, M=7 is NaN. */
float oracle_e4m3_decode(uint8_t code)
{
    int sign = code >> 7;
    int E = (code >> 3) & 0xF;
    int M = code & 0x7;
    float v;
    if (E == 15 && M == 7)
        return NAN;
    if (E == 0)
        v = ldexpf((float)M, -9);           /* (M/8) * 2^-6 */
    else
        v = ldexpf((float)(8 + M), E - 10); /* (1 + M/8) * 2^(E-7) */
    return sign ? -v : v;
}

/* Encode one FP32 value to E4M3: round to nearest, ties to even code,
 * subnormals kept, |y| >= 448 saturates to 448, NaN -> 0x7F | sign.
 * Works on the FP32 bit pattern only. */
uint8_t oracle_e4m3_encode(float y)
{
    uint32_t u;
    memcpy(&u, &y, 4);
    uint8_t sign = (uint8_t)((u >> 24) & 0x80);
    uint32_t a = u & 0x7FFFFFFFu;
    if (a > 0x7F800000u)               /* NaN */
        return sign | 0x7F;
    if (a >= 0x43E00000u)              /* |y| >= 448 (and inf): saturate */
        return sign | 0x7E;
    if (a == 0)
        return sign;
    int e = (int)(a >> 23) - 127;      /* unbiased exponent; a is normal or
                                          FP32-subnormal (then e = -127) */
    if (e >= -6) {
        /* E4M3 normal binade [2^e, 2^(e+1)): keep 3 of the 23 mantissa bits,
         * round the dropped 20 bits to nearest, ties to even. */
        uint32_t mant = a & 0x7FFFFFu;
        uint32_t keep = mant >> 20;
        uint32_t rest = mant & 0xFFFFFu;
        const uint32_t half = 0x80000u;
        if (rest > half || (rest == half && (keep & 1u)))
            keep++;
        int E = e + 7;
        if (keep == 8) {               /* mantissa carry into the exponent */
            keep = 0;
            E++;
        }
        return sign | (uint8_t)((E << 3) | keep);
    }
    /* Below the smallest normal 2^-6: the grid is uniform with step 2^-9, so
     * the code is the integer nearest |y| * 2^9 (exact multiply), ties to
     * even.  n == 8 is the smallest normal, code 0x08. */
    {
        float v = fabsf(y) * 512.0f;
        uint32_t n = (uint32_t)v;      /* truncation; v < 8 */
        float frac = v - (float)n;     /* exact */
        if (frac > 0.5f || (frac == 0.5f && (n & 1u)))
            n++;
        return sign | (uint8_t)n;
    }
}

void oracle_e4m3_encode_array(const float* x, uint8_t* out, int64_t n)
{
    for (int64_t i = 0; i < n; i++)
        out[i] = oracle_e4m3_encode(x[i]);
}

void oracle_e4m3_decode_array(const uint8_t* x, float* out, int64_t n)
{
    for (int64_t i = 0; i < n; i++)
        out[i] = oracle_e4m3_decode(x[i]);
}

/* ------------------------------------------------------------------------- */
/* Algorithm 1, one query row                                                 */
/* ------------------------------------------------------------------------- */

enum { ORDER_FORWARD = 0, ORDER_REVERSE = 1 };
enum { CAST_NONE = 0, CAST_E4M3 = 1 };
enum { SCALE_STATIC = 0, SCALE_DYNAMIC = 1 };

typedef struct {
    const float* q;     /* [B][Hq][N][d]  */
    const float* k;     /* [B][Hkv][N][d] */
    const float* v;     /* [B][Hkv][N][d] */
    float* out;         /* [n_rows][d]    */
    float* lse;         /* [n_rows]       (nullable) */
    uint32_t* counts;   /* [n_rows][3]    (nullable) */
    int B, Hq, Hkv, Nq, Nk, d, causal, Bc, order, cast, n_sink;
    int scale_mode, k0;     /* k0 = log2 S (dynamic scale only) */
    float S;
    double qk_descale;  /* q_descale * k_descale (exact in double) */
    float v_descale;
    float* amb;         /* [n_rows][d] code-ambiguity bound (nullable) */
    double amb_rel;     /* relative half-width of the ambiguity window */
    double jitter_rel;  /* planted exp2 error (test build only; else 0) */
    uint32_t* gap_hist; /* [B*Hq][nblk_all][nbins] (nullable) */
    uint32_t* blk_zero; /* [B*Hq][nblk_all] (nullable with gap_hist) */
    int nbins, nblk_all;
    const int64_t* rows;/* flat (b*Hq + hq)*N + r, n_rows of them */
    int64_t n_rows;
    int nthreads;
    int64_t next;       /* work counter */
    pthread_mutex_t lock;
} attn_job;

#ifdef ORACLE_TEST_PLANTS
/* Test build only (liboracle_plant.so, -DORACLE_TEST_PLANTS): a planted exp2
 * error, so that the code-ambiguity bound can be checked against a known
 * perturbation.  splitmix64 finaliser: a fixed hash of (row, key). */
static uint64_t mix64(uint64_t z)
{
    z += 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

static double planted_exp2_error(const attn_job* J, int64_t flat, int key)
{
    const uint64_t h = mix64(((uint64_t)flat << 32) ^ (uint64_t)key);
    return 1.0 + J->jitter_rel * (2.0 * ((double)(h >> 11) * 0x1p-53) - 1.0);
}
#endif

static void attn_row(const attn_job* J, int64_t flat, float* out_row,
                     float* lse_row, uint32_t* cnt_row, float* amb_row, float* D,
                     float* P, float* F, float* o, float* blk, float* a, float* ablk)
{
    const int Nq = J->Nq, Nk = J->Nk, d = J->d, Bc = J->Bc;
    const int64_t bh = flat / Nq;
    const int r = (int)(flat % Nq);
    const int b = (int)(bh / J->Hq), hq = (int)(bh % J->Hq);
    const int hk = hq / (J->Hq / J->Hkv);
    const float* qr = J->q + flat * (int64_t)d;
    const float* K = J->k + ((int64_t)b * J->Hkv + hk) * (int64_t)Nk * d;
    const float* V = J->v + ((int64_t)b * J->Hkv + hk) * (int64_t)Nk * d;
    const float S = J->S;
    /* exp(z) with z = D qd kd / sqrt(d) is exp2(D * c), D the raw dot of the
     * stored values and qd, kd the per-tensor descales of the QKV
     * quantization (Sec. 6.1); c rounded once from double */
    const float c = (float)(1.4426950408889634074 * J->qk_descale / sqrt((double)d));

    /* query row r sits at key position Nk - Nq + r: the Nq queries are the
     * last Nq positions of a sequence whose Nk keys are all cached (Nq = Nk:
     * plain self-attention); under causal masking the row sees keys up to
     * its own position, otherwise all Nk */
    const int L = J->causal ? Nk - Nq + r + 1 : Nk;    /* valid keys 0..L-1 */
    const int nblk = (L + Bc - 1) / Bc;

    /* running state of the row, FP32: maximum of the raw dots (and its
     * scaled copy mc = fl(m c)), the pre-cast sum l and the accumulator o */
    float m = -INFINITY, mc = -INFINITY, ell = 0.0f;
    for (int i = 0; i < d; i++)
        o[i] = a[i] = 0.0f;
    if (cnt_row)
        cnt_row[0] = cnt_row[1] = cnt_row[2] = 0;

    for (int it = 0; it < nblk; it++) {
        /* blocks in ascending order, or descending for the reverse order */
        const int j = (J->order == ORDER_FORWARD) ? it : nblk - 1 - it;
        const int t0 = j * Bc;
        const int t1 = (t0 + Bc < L) ? t0 + Bc : L;
        const int nt = t1 - t0;

        /* scores: raw dot products, rounded once to FP32 */
        float mloc = -INFINITY;
        for (int t = 0; t < nt; t++) {
            const float* kt = K + (int64_t)(t0 + t) * d;
            double acc = 0.0;
            for (int i = 0; i < d; i++)
                acc += (double)qr[i] * (double)kt[i];
            D[t] = (float)acc;
            if (D[t] > mloc)
                mloc = D[t];
        }
        /* new running maximum; the rescale factor of the old state is the
         * base-2 exponential of the difference of the scaled maxima (1
         * exactly when the maximum does not move, 0 on the first block) */
        const float m_new = (m > mloc) ? m : mloc;
        const float mc_new = m_new * c;
        const float alpha = (float)exp2((double)(mc - mc_new));

        /* per-block diagnostic: the gap g = -(block's largest exponent
         * argument), so the block's largest P is 2^-g; binned by floor */
        if (J->gap_hist) {
            const double g = floor(-(double)fmaf(mloc, c, -mc_new));
            const int bin = g <= 0.0 ? 0 : (g >= J->nbins - 1 ? J->nbins - 1 : (int)g);
            __atomic_fetch_add(&J->gap_hist[((int64_t)bh * J->nblk_all + j) * J->nbins + bin],
                               1u, __ATOMIC_RELAXED);
        }

        /* P of every key in FP32 (exp2 in double, rounded once); the sum l
         * takes these pre-cast values (Sec. 6.1) */
        float psum = 0.0f;
        for (int t = 0; t < nt; t++) {
            const float x = fmaf(D[t], c, -mc_new);
            double e = exp2((double)x);
#ifdef ORACLE_TEST_PLANTS
            if (J->jitter_rel != 0.0)
                e *= planted_exp2_error(J, flat, t0 + t);
#endif
            P[t] = (float)e;
            psum += P[t];
        }
        ell = alpha * ell + psum;

        /* scale of this block's cast: S, or with the dynamic scale 2^kj
         * chosen from the block's largest exponent argument */
        float Sj = S;
        int back = 0;                           /* S units = block units * 2^back */
        if (J->scale_mode == SCALE_DYNAMIC) {
            const float xmax = fmaf(mloc, c, -mc_new);
            const double f = floor(-(double)xmax);
            int kj = J->k0 + (f > 0.0 ? (f > 200.0 ? 200 : (int)f) : 0);
            if (kj > 126)
                kj = 126;
            Sj = ldexpf(1.0f, kj);
            back = J->k0 - kj;
        }

        /* the cast: E4M3 code of P * Sj; zero codes are counted per key
         * category (Prop. 1); the decoded value goes back to S units */
        for (int t = 0; t < nt; t++) {
            const float y = P[t] * Sj;
            F[t] = 0.0f;
            if (J->cast == CAST_E4M3) {
                const uint8_t e = oracle_e4m3_encode(y);
                if (amb_row) {
                    /* codes reachable from any y' within amb_rel of y: the
                     * cast is monotone, so the two ends bound them */
                    const uint8_t lo = oracle_e4m3_encode((float)((double)y * (1.0 - J->amb_rel)));
                    const uint8_t hi = oracle_e4m3_encode((float)((double)y * (1.0 + J->amb_rel)));
                    F[t] = ldexpf(oracle_e4m3_decode(hi) - oracle_e4m3_decode(lo), back);
                }
                if (cnt_row && e == 0x00) {
                    const int key = t0 + t;
                    const int cat = key < J->n_sink ? 0 : (key < Bc ? 1 : 2);
                    cnt_row[cat]++;
                }
                if (J->blk_zero && e == 0x00)
                    __atomic_fetch_add(&J->blk_zero[(int64_t)bh * J->nblk_all + j], 1u,
                                       __ATOMIC_RELAXED);
                P[t] = ldexpf(oracle_e4m3_decode(e), back);
            } else {
                P[t] = ldexpf(y, back);
            }
        }

        /* the accumulator takes the cast values (Sec. 6.1): FP32 sum of this
         * block's P~ v, added to the rescaled old accumulator */
        for (int i = 0; i < d; i++)
            blk[i] = 0.0f;
        for (int t = 0; t < nt; t++) {
            const float* vt = V + (int64_t)(t0 + t) * d;
            for (int i = 0; i < d; i++)
                blk[i] += P[t] * vt[i];
        }
        for (int i = 0; i < d; i++)
            o[i] = alpha * o[i] + blk[i];
        if (amb_row) {
            /* the same recurrence over |V| and the code spans */
            for (int i = 0; i < d; i++)
                ablk[i] = 0.0f;
            for (int t = 0; t < nt; t++) {
                const float* vt = V + (int64_t)(t0 + t) * d;
                for (int i = 0; i < d; i++)
                    ablk[i] += F[t] * fabsf(vt[i]);
            }
            for (int i = 0; i < d; i++)
                a[i] = alpha * a[i] + ablk[i];
        }

        m = m_new;
        mc = mc_new;
    }

    /* the output divides by S and by the pre-cast sum; lse is the
     * natural-log log-sum-exp of z */
    const float denom = S * ell;
    for (int i = 0; i < d; i++)
        out_row[i] = o[i] / denom * J->v_descale;
    if (amb_row)
        for (int i = 0; i < d; i++)
            amb_row[i] = a[i] / denom * J->v_descale;
    if (lse_row)
        *lse_row = (float)(((double)mc + log2((double)ell)) * 0.6931471805599453094);
}

static void* attn_worker(void* arg)
{
    attn_job* J = (attn_job*)arg;
    const int d = J->d, Bc = J->Bc;
    float* D = (float*)malloc(sizeof(float) * (size_t)Bc);
    float* P = (float*)malloc(sizeof(float) * (size_t)Bc);
    float* F = (float*)malloc(sizeof(float) * (size_t)Bc);
    float* o = (float*)malloc(sizeof(float) * (size_t)d);
    float* blk = (float*)malloc(sizeof(float) * (size_t)d);
    float* a = (float*)malloc(sizeof(float) * (size_t)d);
    float* ablk = (float*)malloc(sizeof(float) * (size_t)d);
    for (;;) {
        int64_t i;
        pthread_mutex_lock(&J->lock);
        i = J->next++;
        pthread_mutex_unlock(&J->lock);
        if (i >= J->n_rows)
            break;
        const int64_t flat = J->rows ? J->rows[i] : i;
        attn_row(J, flat, J->out + i * (int64_t)d, J->lse ? J->lse + i : NULL,
                 J->counts ? J->counts + 3 * i : NULL, J->amb ? J->amb + i * (int64_t)d : NULL,
                 D, P, F, o, blk, a, ablk);
    }
    free(D);
    free(P);
    free(F);
    free(o);
    free(blk);
    free(a);
    free(ablk);
    return NULL;
}

static int run_threads(void* (*fn)(void*), void* job, pthread_mutex_t* lock,
                       int nthreads)
{
    if (nthreads < 1)
        nthreads = 1;
    if (nthreads > 256)
        nthreads = 256;
    pthread_t th[256];
    pthread_mutex_init(lock, NULL);
    int started = 0;
    for (int i = 0; i < nthreads; i++) {
        if (pthread_create(&th[i], NULL, fn, job) != 0)
            break;
        started++;
    }
    if (started == 0)
        fn(job);
    for (int i = 0; i < started; i++)
        pthread_join(th[i], NULL);
    pthread_mutex_destroy(lock);
    return 0;
}

/*
 * Algorithm 1 on a list of query rows.
 *   q: [B][Hq][N][d], k, v: [B][Hkv][N][d], all FP32 host arrays holding the
 *   exact values the device consumed.
 *   rows: flat row ids (b*Hq + hq)*N + r (NULL = all B*Hq*N rows in order).
 *   out: [n_rows][d], lse: [n_rows] (nullable), counts: [n_rows][3]
 *   (nullable; categories key < n_sink, n_sink <= key < Bc, key >= Bc).
 *   cast: 0 = no cast (P*S used as is), 1 = E4M3.
 *   scale_mode: 0 = static S, 1 = dynamic per-block 2^kj (S must be 2^k0,
 *   0 <= k0 <= 8).
 *   amb: [n_rows][d] (nullable), the code-ambiguity bound.  An implementation
 *   whose exp2 is within a few ulps of the correctly rounded one may land a
 *   P*S value that sits next to an E4M3 rounding midpoint on the other code.
 *   amb[i] bounds what every such choice can move out[i]: with y = P*S and
 *   F = decode(cast(y (1 + amb_rel))) - decode(cast(y (1 - amb_rel))) (zero
 *   unless y lies within amb_rel of a midpoint), it runs the same recurrence
 *   as O over F |V| and takes the same epilogue.  Both ends come from the
 *   cast above, which is monotone in y.
 *   jitter_rel: must be 0, except in the test build compiled with
 *   -DORACLE_TEST_PLANTS, where each exp2 of a P value is multiplied by
 *   1 + jitter_rel * u, u in [-1, 1) a fixed hash of (row, key), to check
 *   amb against a known perturbation.
 *   gap_hist, blk_zero, nbins: the per-block diagnostic (both nullable, both
 *   or neither; 1 <= nbins <= 64), accumulated over the given rows and zeroed
 *   here first.  gap_hist[bh][j][bin] counts the rows that visit block j
 *   with bin = min(max(floor(g), 0), nbins - 1), g = -fma(block max, c, -mc)
 *   (the row's block maximum of the raw dots, mc = fl(m_new c) after the
 *   block), i.e. the block's largest P is 2^-g: the multi-sink form of the
 *   sink gap (Limitations and Future Work, "Multi-sink patterns").
 *   blk_zero[bh][j] counts block j's zero codes over the rows (Prop. 1).
 *   Both are [B*Hq][ceil(N/block_kv)](...) with bh = b*Hq + hq.
 * Returns 0, or -1 on an invalid argument.
 */
int oracle_attn_full(const float* q, const float* k, const float* v, float* out,
                     float* lse, uint32_t* counts, float* amb, uint32_t* gap_hist,
                     uint32_t* blk_zero, int nbins, int B, int Hq, int Hkv, int Nq, int Nk,
                     int d, int causal, int block_kv, int order, float S, int cast,
                     int scale_mode, int n_sink, float q_descale, float k_descale,
                     float v_descale, double amb_rel, double jitter_rel, const int64_t* rows,
                     int64_t n_rows, int nthreads)
{
    const int N = Nq;           /* rows are indexed over the Nq queries */
    if (Nq > Nk)
        return -1;
    if (!(amb_rel >= 0.0) || !(amb_rel < 0.5) || !(fabs(jitter_rel) < 0.5))
        return -1;
#ifndef ORACLE_TEST_PLANTS
    if (jitter_rel != 0.0)
        return -1;              /* the plant exists only in the test build */
#endif
    if ((gap_hist != NULL) != (blk_zero != NULL) || (gap_hist && (nbins < 1 || nbins > 64)))
        return -1;
    if (!q || !k || !v || !out || B < 1 || Hq < 1 || Hkv < 1 || N < 1 ||
        d < 1 || Hq % Hkv != 0 || block_kv < 1 || !(S > 0.0f) ||
        !isfinite(S) || (order != 0 && order != 1) || (cast != 0 && cast != 1) ||
        (scale_mode != 0 && scale_mode != 1) || n_sink < 0 || n_rows < 0 ||
        !(q_descale > 0.0f) || !(k_descale > 0.0f) || !(v_descale > 0.0f) ||
        !isfinite(q_descale) || !isfinite(k_descale) || !isfinite(v_descale))
        return -1;
    int k0 = 0;
    if (scale_mode == SCALE_DYNAMIC) {
        int e;
        const float f = frexpf(S, &e);          /* S = f * 2^e, f in [0.5, 1) */
        k0 = e - 1;
        if (f != 0.5f || k0 < 0 || k0 > 8)
            return -1;
    }
    if (rows)
        for (int64_t i = 0; i < n_rows; i++)
            if (rows[i] < 0 || rows[i] >= (int64_t)B * Hq * N)
                return -1;
    if (!rows && n_rows != (int64_t)B * Hq * N)
        return -1;
    attn_job J;
    memset(&J, 0, sizeof(J));
    J.q = q; J.k = k; J.v = v; J.out = out; J.lse = lse; J.counts = counts;
    J.B = B; J.Hq = Hq; J.Hkv = Hkv; J.Nq = Nq; J.Nk = Nk; J.d = d; J.causal = causal;
    J.Bc = block_kv; J.order = order; J.cast = cast; J.n_sink = n_sink;
    J.scale_mode = scale_mode; J.k0 = k0;
    J.S = S; J.rows = rows; J.n_rows = n_rows; J.nthreads = nthreads;
    J.qk_descale = (double)q_descale * (double)k_descale;
    J.v_descale = v_descale;
    J.amb = amb;
    J.amb_rel = amb_rel;
    J.jitter_rel = jitter_rel;
    J.gap_hist = gap_hist;
    J.blk_zero = blk_zero;
    J.nbins = nbins;
    J.nblk_all = (Nk + block_kv - 1) / block_kv;
    if (gap_hist) {
        memset(gap_hist, 0, sizeof(uint32_t) * (size_t)B * Hq * J.nblk_all * nbins);
        memset(blk_zero, 0, sizeof(uint32_t) * (size_t)B * Hq * J.nblk_all);
    }
    run_threads(attn_worker, &J, &J.lock, nthreads);
    return 0;
}

/* ------------------------------------------------------------------------- */
/* Textbook softmax attention in FP64 (no blocks, no cast): the reference the */
/* MSE is measured against.                                                   */
/* ------------------------------------------------------------------------- */

typedef struct {
    const float *q, *k, *v;
    double* out;
    double* lse;
    int B, Hq, Hkv, Nq, Nk, d, causal;
    double qk_descale, v_descale;
    const int64_t* rows;
    int64_t n_rows, next;
    pthread_mutex_t lock;
} ref_job;

static void* ref_worker(void* arg)
{
    ref_job* J = (ref_job*)arg;
    const int Nq = J->Nq, Nk = J->Nk, d = J->d;
    double* z = (double*)malloc(sizeof(double) * (size_t)Nk);
    for (;;) {
        int64_t i;
        pthread_mutex_lock(&J->lock);
        i = J->next++;
        pthread_mutex_unlock(&J->lock);
        if (i >= J->n_rows)
            break;
        const int64_t flat = J->rows ? J->rows[i] : i;
        const int64_t bh = flat / Nq;
        const int r = (int)(flat % Nq);
        const int b = (int)(bh / J->Hq), hq = (int)(bh % J->Hq);
        const int hk = hq / (J->Hq / J->Hkv);
        const float* qr = J->q + flat * (int64_t)d;
        const float* K = J->k + ((int64_t)b * J->Hkv + hk) * (int64_t)Nk * d;
        const float* V = J->v + ((int64_t)b * J->Hkv + hk) * (int64_t)Nk * d;
        const int L = J->causal ? Nk - Nq + r + 1 : Nk;   /* row r at position Nk - Nq + r */
        const double scale = J->qk_descale / sqrt((double)d);
        double zmax = -INFINITY;
        for (int t = 0; t < L; t++) {
            double acc = 0.0;
            for (int c = 0; c < d; c++)
                acc += (double)qr[c] * (double)K[(int64_t)t * d + c];
            z[t] = acc * scale;
            if (z[t] > zmax)
                zmax = z[t];
        }
        double ell = 0.0;
        for (int t = 0; t < L; t++) {
            z[t] = exp(z[t] - zmax);
            ell += z[t];
        }
        double* o = J->out + i * (int64_t)d;
        for (int c = 0; c < d; c++)
            o[c] = 0.0;
        for (int t = 0; t < L; t++)
            for (int c = 0; c < d; c++)
                o[c] += z[t] * (double)V[(int64_t)t * d + c];
        for (int c = 0; c < d; c++)
            o[c] = o[c] / ell * J->v_descale;
        if (J->lse)
            J->lse[i] = zmax + log(ell);
    }
    free(z);
    return NULL;
}

int oracle_ref_fp64_kv(const float* q, const float* k, const float* v, double* out,
                       double* lse, int B, int Hq, int Hkv, int Nq, int Nk, int d, int causal,
                       double q_descale, double k_descale, double v_descale,
                       const int64_t* rows, int64_t n_rows, int nthreads)
{
    const int N = Nq;
    if (!q || !k || !v || !out || B < 1 || Hq < 1 || Hkv < 1 || Nq < 1 || Nk < Nq ||
        d < 1 || Hq % Hkv != 0 || n_rows < 0)
        return -1;
    if (rows)
        for (int64_t i = 0; i < n_rows; i++)
            if (rows[i] < 0 || rows[i] >= (int64_t)B * Hq * N)
                return -1;
    if (!rows && n_rows != (int64_t)B * Hq * N)
        return -1;
    ref_job J;
    memset(&J, 0, sizeof(J));
    J.q = q; J.k = k; J.v = v; J.out = out; J.lse = lse;
    J.B = B; J.Hq = Hq; J.Hkv = Hkv; J.Nq = Nq; J.Nk = Nk; J.d = d; J.causal = causal;
    J.rows = rows; J.n_rows = n_rows;
    J.qk_descale = q_descale * k_descale;
    J.v_descale = v_descale;
    run_threads(ref_worker, &J, &J.lock, nthreads);
    return 0;
}

int oracle_version(void) { return ORACLE_VERSION; }
