/*
 * Reference oracle for the W4A8 (Q4_0 weight x Q8_0 activation) MoE hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, plain, obviously-correct
 * CPU definition that the HIP library is checked against.  Only the tests, the
 * smoke check and the CPU-baseline leg of the benchmark may load it; the
 * product library never does, and it shares no code, header, table or helper
 * with the HIP sources.
 *
 * Build: gcc -std=c11 -O2 -ffp-contract=off -fopenmp -fPIC -shared
 *   (no fast-math, no SIMD intrinsics, no FMA contraction: every fp32 step
 *    below is one IEEE-754 binary32 operation, every fp64 step one binary64
 *    operation).
 *
 * What the paper fixes and what is a stated reading (see the design notes):
 *  - Weights: group-wise symmetric 4-bit "Q4_0 family" blocks, two values per
 *    byte, one scale per group (Sec. 2.3 "Weight quantization").  Reading: 32
 *    weights per block, fp16 scale d = m / -8 where m is the signed element of
 *    largest magnitude (first index on ties), value (q - 8) * d with q in
 *    0..15; 18-byte block = fp16 d then 16 bytes, byte j holding element j in
 *    the low nibble and element j+16 in the high nibble.
 *  - Activations: quantized per group to 8 bits with a scale (Sec. 3.3 "CPU
 *    decode: W4A8").  Reading: 32 per block, fp16 d = amax/127, codes
 *    round-half-away-from-zero of x / d against the stored (rounded) scale,
 *    clamped to +-127; 34-byte block = fp16 d then 32 int8.
 *  - Dot product: integer multiply-adds of the 4-bit weight codes with the
 *    8-bit activation codes, then scaling (Sec. 3.3; the Q4_0 x Q8_0 scheme
 *    named in Sec. 1, contribution 2).
 *  - MoE FFN: routed top-k experts plus one always-on shared expert
 *    (Sec. 2.2 "The model"), all routed token-expert pairs of a layer in one
 *    grouped pass (Sec. 3.2 "GPU prefill").  Reading: expert MLP is
 *    down(SiLU(gate x) * (up x)), gate rows first in the fused gate/up matrix,
 *    shared expert with weight 1, x quantized once per token, h quantized per
 *    (token, expert) pair.
 *
 * Parity pins (tests/test_oracle_pins.py) tie each function to something other
 * than itself: numpy's fp16 conversion, the Q8_0 round-trip bound
 * |x - q d| <= d/2, brute-force code search, hand-built blocks, the fp64
 * dequantize-then-matmul definition, the textbook SwiGLU MLP and special
 * routing cases.  The SiLU ulp level of the GPU and its summation order are
 * "parity unpinned": they are covered by the float tolerance only.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define QK 32          /* elements per quantization block           */
#define Q4_BYTES 18    /* fp16 scale + 16 bytes of packed nibbles    */
#define Q8_BYTES 34    /* fp16 scale + 32 signed bytes               */

/* ------------------------------------------------------------------ */
/* IEEE-754 binary16 <-> binary32, written from the format definition. */
/* ------------------------------------------------------------------ */

/* binary32 -> binary16, round to nearest, ties to even; subnormals kept;
 * overflow to +-inf; NaN stays NaN (quiet). */
uint16_t orc_f32_to_f16(float f)
{
    uint32_t x;
    memcpy(&x, &f, 4);
    uint32_t sign = (x >> 16) & 0x8000u;
    uint32_t ax = x & 0x7FFFFFFFu;
    if (ax >= 0x7F800000u)                       /* inf or NaN */
        return (uint16_t)(sign | 0x7C00u | (ax > 0x7F800000u ? 0x0200u : 0u));
    if (ax >= 0x477FF000u)                       /* >= 65520: rounds to inf */
        return (uint16_t)(sign | 0x7C00u);
    if (ax < 0x38800000u) {                      /* below 2^-14: half subnormal */
        if (ax < 0x33000000u)                    /* < 2^-25 (tie at 2^-25 -> 0) */
            return (uint16_t)sign;
        uint32_t e = ax >> 23;                   /* 102..112 */
        uint32_t m = (ax & 0x7FFFFFu) | 0x800000u;
        uint32_t shift = 126u - e;               /* 14..24 */
        uint32_t q = m >> shift;
        uint32_t rem = m & ((1u << shift) - 1u);
        uint32_t half = 1u << (shift - 1u);
        if (rem > half || (rem == half && (q & 1u)))
            q++;
        return (uint16_t)(sign | q);
    }
    uint32_t e = (ax >> 23) - 127u + 15u;
    uint32_t m = ax & 0x7FFFFFu;
    uint32_t q = (e << 10) | (m >> 13);
    uint32_t rem = m & 0x1FFFu;
    if (rem > 0x1000u || (rem == 0x1000u && (q & 1u)))
        q++;                                      /* carry into exponent is correct */
    return (uint16_t)(sign | q);
}

/* binary16 -> binary32, exact. */
float orc_f16_to_f32(uint16_t h)
{
    uint32_t sign = ((uint32_t)h & 0x8000u) << 16;
    uint32_t e = ((uint32_t)h >> 10) & 0x1Fu;
    uint32_t m = (uint32_t)h & 0x3FFu;
    uint32_t x;
    if (e == 0x1Fu) {
        x = sign | 0x7F800000u | (m << 13);
    } else if (e != 0) {
        x = sign | ((e - 15u + 127u) << 23) | (m << 13);
    } else if (m == 0) {
        x = sign;
    } else {                                      /* subnormal: m * 2^-24 */
        float v = (float)m * (1.0f / 16777216.0f);   /* exact: power-of-two scale */
        memcpy(&x, &v, 4);
        x |= sign;
    }
    float f;
    memcpy(&f, &x, 4);
    return f;
}

static uint16_t rd16(const uint8_t *p) { return (uint16_t)(p[0] | (p[1] << 8)); }
static void wr16(uint8_t *p, uint16_t v) { p[0] = (uint8_t)(v & 0xFF); p[1] = (uint8_t)(v >> 8); }

/* ------------------------------------------------------------------ */
/* Q8_0 activation quantization (Sec. 3.3: per-group 8-bit + scale).   */
/* ------------------------------------------------------------------ */

/* One block of 32 fp32 values -> 34 bytes.  Every step is one fp32 op:
 * amax exact; d32 = amax / 127 (one correctly rounded division); the stored
 * scale is fp16(d32) (RNE); codes are round-half-away(x * (1 / d_stored))
 * clamped to +-127; a zero stored scale gives all-zero codes. */
void orc_q8_0_block(const float *x, uint8_t *out)
{
    float amax = 0.0f;
    for (int i = 0; i < QK; i++) {
        float a = fabsf(x[i]);
        if (a > amax) amax = a;
    }
    float d32 = amax / 127.0f;
    uint16_t d16 = orc_f32_to_f16(d32);
    float df = orc_f16_to_f32(d16);
    wr16(out, d16);
    if (df == 0.0f) {
        memset(out + 2, 0, QK);
        return;
    }
    float id = 1.0f / df;
    for (int i = 0; i < QK; i++) {
        float v = x[i] * id;
        float r = roundf(v);                  /* half away from zero */
        int q = (int)r;
        if (q > 127) q = 127;
        if (q < -127) q = -127;
        out[2 + i] = (uint8_t)(int8_t)q;
    }
}

void orc_q8_0_quantize(const float *x, uint8_t *out, int64_t rows, int64_t K)
{
    int64_t nb = K / QK;
    #pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < rows; r++)
        for (int64_t b = 0; b < nb; b++)
            orc_q8_0_block(x + r * K + b * QK, out + (r * nb + b) * Q8_BYTES);
}

/* ------------------------------------------------------------------ */
/* Q4_0 weight quantization (Sec. 2.3, read as d = m / -8).            */
/* ------------------------------------------------------------------ */

void orc_q4_0_block(const float *w, uint8_t *out)
{
    float m = 0.0f, amax = 0.0f;
    for (int i = 0; i < QK; i++) {          /* first index of largest |w| */
        float a = fabsf(w[i]);
        if (a > amax) { amax = a; m = w[i]; }
    }
    float d32 = m / -8.0f;
    uint16_t d16 = orc_f32_to_f16(d32);
    float df = orc_f16_to_f32(d16);
    float id = (df != 0.0f) ? 1.0f / df : 0.0f;
    int q[QK];
    for (int i = 0; i < QK; i++) {
        float p = w[i] * id;                  /* one fp32 multiply   */
        float v = p + 8.5f;                   /* one fp32 add        */
        int qi = (int)floorf(v);
        if (qi > 15) qi = 15;
        if (qi < 0) qi = 0;                   /* reachable only with an fp16-subnormal scale */
        q[i] = qi;
    }
    wr16(out, d16);
    for (int j = 0; j < 16; j++)
        out[2 + j] = (uint8_t)(q[j] | (q[j + 16] << 4));
}

void orc_q4_0_quantize(const float *w, uint8_t *out, int64_t rows, int64_t K)
{
    int64_t nb = K / QK;
    #pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < rows; r++)
        for (int64_t b = 0; b < nb; b++)
            orc_q4_0_block(w + r * K + b * QK, out + (r * nb + b) * Q4_BYTES);
}

/* ------------------------------------------------------------------ */
/* Integer block dot and the W4A8 matrix-vector product (Sec. 3.3).    */
/* ------------------------------------------------------------------ */

/* s = sum_i (q_w,i - 8) * q_a,i over one block, exact in int32. */
int32_t orc_blockdot(const uint8_t *wb, const uint8_t *ab)
{
    const int8_t *qa = (const int8_t *)(ab + 2);
    int32_t s = 0;
    for (int j = 0; j < 16; j++) {
        int lo = (wb[2 + j] & 0x0F) - 8;       /* element j      */
        int hi = (wb[2 + j] >> 4) - 8;         /* element j + 16 */
        s += lo * qa[j] + hi * qa[j + 16];
    }
    return s;
}

/* y[n] = sum_b d_w[n,b] * d_a[b] * s[n,b], each term exact in fp64 and summed
 * in block order in fp64 (left unrounded); R[n] = sum_b |term|.  Either output
 * pointer may be NULL. */
void orc_gemv(const uint8_t *w, const uint8_t *xq, int64_t N, int64_t K,
              double *y, double *R)
{
    int64_t nb = K / QK;
    #pragma omp parallel for schedule(static)
    for (int64_t n = 0; n < N; n++) {
        double acc = 0.0, mag = 0.0;
        for (int64_t b = 0; b < nb; b++) {
            const uint8_t *wb = w + (n * nb + b) * Q4_BYTES;
            const uint8_t *ab = xq + b * Q8_BYTES;
            double t = (double)orc_f16_to_f32(rd16(wb)) *
                       (double)orc_f16_to_f32(rd16(ab)) *
                       (double)orc_blockdot(wb, ab);
            acc += t;
            mag += fabs(t);
        }
        if (y) y[n] = acc;
        if (R) R[n] = mag;
    }
}

/* Independent cross-check of orc_gemv: dequantize every factor to fp64 and
 * take the plain dot product over k, y[n] = sum_k ((q_w-8) d_w) * (q_a d_a). */
void orc_gemv_dequant(const uint8_t *w, const uint8_t *xq, int64_t N, int64_t K,
                      double *y)
{
    int64_t nb = K / QK;
    #pragma omp parallel for schedule(static)
    for (int64_t n = 0; n < N; n++) {
        double acc = 0.0;
        for (int64_t k = 0; k < K; k++) {
            int64_t b = k / QK, i = k % QK;
            const uint8_t *wb = w + (n * nb + b) * Q4_BYTES;
            const uint8_t *ab = xq + b * Q8_BYTES;
            int nib = (i < 16) ? (wb[2 + i] & 0x0F) : (wb[2 + i - 16] >> 4);
            double wv = (double)(nib - 8) * (double)orc_f16_to_f32(rd16(wb));
            double av = (double)((const int8_t *)(ab + 2))[i] * (double)orc_f16_to_f32(rd16(ab));
            acc += wv * av;
        }
        y[n] = acc;
    }
}

/* ------------------------------------------------------------------ */
/* The routed + shared MoE FFN layer (Sec. 2.2, Sec. 3.2, Sec. 3.3).   */
/* ------------------------------------------------------------------ */

static double silu_d(double g) { return g / (1.0 + exp(-g)); }

/*
 * Pair numbering: routed slot j of token t is pair t*k + j; the shared
 * expert's pair for token t is T*k + t.  Per-pair outputs are indexed by it.
 *
 * For every token t:
 *   xq      = Q8_0(hidden[t])
 *   for every slot j with e = ids[t,j] >= 0, and for the shared expert:
 *     gu    = fp32( W4A8 gemv of W_gu[e] with xq )              (2I values)
 *     h     = fp32( silu(gu[0:I]) * gu[I:2I] ), evaluated in fp64
 *     hq    = Q8_0(h)                (or hq_in for the pair, when given)
 *     y     = W4A8 gemv of W_d[e] with hq  (fp64, unrounded)
 *   out[t]  = sum_j w[t,j] * y_j + s[t] * y_shared, accumulated in fp64
 *   R[t]    = sum_j |w[t,j]| * R_y_j + |s[t]| * R_y_shared
 * s[t] = shared_w[t] when shared_w is given (the sigmoid gate of a gated
 * shared expert, evaluated by the caller), else 1 (always on, Sec. 2.2).
 *
 * hq_in (may be NULL): Q8_0 codes to use for h, one 34-byte block row per pair
 * (a choice among results the oracle itself accepts; see the tests).
 * Optional outputs (NULL to skip): gu_out [P][2I] fp32, Rgu_out [P][2I] fp64,
 * h_out [P][I] fp32, hq_out [P][I/32] blocks; out, R [T][H] fp64 are required.
 * Slots with id < 0 contribute nothing and leave their pair rows untouched.
 * Returns 0, or -1 if an id is >= E.
 */
int orc_moe(const float *hidden, const int32_t *ids, const float *wts,
            const uint8_t *w_gu, const uint8_t *w_d,
            const uint8_t *ws_gu, const uint8_t *ws_d,
            int64_t T, int64_t H, int64_t I, int64_t E, int64_t k,
            const uint8_t *hq_in,
            double *out, double *R,
            float *gu_out, double *Rgu_out, float *h_out, uint8_t *hq_out,
            const double *shared_w)
{
    int64_t nbH = H / QK, nbI = I / QK;
    size_t gu_bytes = (size_t)(2 * I) * nbH * Q4_BYTES;    /* one expert's gate/up */
    size_t d_bytes = (size_t)H * nbI * Q4_BYTES;           /* one expert's down    */
    for (int64_t i = 0; i < T * k; i++)
        if (ids[i] >= E) return -1;

    int bad = 0;
    #pragma omp parallel for schedule(dynamic, 1)
    for (int64_t t = 0; t < T; t++) {
        uint8_t *xq = malloc((size_t)nbH * Q8_BYTES);
        uint8_t *hq = malloc((size_t)nbI * Q8_BYTES);
        double *gu = malloc(sizeof(double) * 2 * I);
        double *rgu = malloc(sizeof(double) * 2 * I);
        float *h = malloc(sizeof(float) * I);
        double *y = malloc(sizeof(double) * H);
        double *ry = malloc(sizeof(double) * H);
        if (!xq || !hq || !gu || !rgu || !h || !y || !ry) { bad = 1; goto done; }

        orc_q8_0_quantize(hidden + t * H, xq, 1, H);
        for (int64_t n = 0; n < H; n++) { out[t * H + n] = 0.0; R[t * H + n] = 0.0; }

        for (int64_t j = 0; j <= k; j++) {
            const uint8_t *Wgu, *Wd;
            double wj;
            int64_t pair;
            if (j < k) {
                int32_t e = ids[t * k + j];
                if (e < 0) continue;
                Wgu = w_gu + (size_t)e * gu_bytes;
                Wd = w_d + (size_t)e * d_bytes;
                wj = (double)wts[t * k + j];
                pair = t * k + j;
            } else {
                if (!ws_gu || !ws_d) continue;
                Wgu = ws_gu;
                Wd = ws_d;
                wj = shared_w ? shared_w[t] : 1.0;
                pair = T * k + t;
            }
            orc_gemv(Wgu, xq, 2 * I, H, gu, rgu);
            for (int64_t i = 0; i < I; i++) {
                float g = (float)gu[i], u = (float)gu[I + i];
                h[i] = (float)(silu_d((double)g) * (double)u);
            }
            if (gu_out) for (int64_t i = 0; i < 2 * I; i++) gu_out[pair * 2 * I + i] = (float)gu[i];
            if (Rgu_out) for (int64_t i = 0; i < 2 * I; i++) Rgu_out[pair * 2 * I + i] = rgu[i];
            if (h_out) memcpy(h_out + pair * I, h, sizeof(float) * I);
            orc_q8_0_quantize(h, hq, 1, I);
            if (hq_out) memcpy(hq_out + pair * nbI * Q8_BYTES, hq, (size_t)nbI * Q8_BYTES);
            const uint8_t *hq_use = hq_in ? hq_in + pair * nbI * Q8_BYTES : hq;
            orc_gemv(Wd, hq_use, H, I, y, ry);
            for (int64_t n = 0; n < H; n++) {
                out[t * H + n] += wj * y[n];
                R[t * H + n] += fabs(wj) * ry[n];
            }
        }
    done:
        free(xq); free(hq); free(gu); free(rgu); free(h); free(y); free(ry);
    }
    return bad ? -2 : 0;
}

/* ------------------------------------------------------------------ */
/* The set of Q8_0 results that are correct for an uncertain input.   */
/* ------------------------------------------------------------------ */

/*
 * When h itself is only known to within +-dh[i] (it comes out of fp32 sums
 * whose order is not fixed by the method), Q8_0(h) is one of a small set of
 * results.  For every block this lists each fp16 scale that some h' in the box
 * |h' - h| <= dh can produce (consecutive fp16 values, nscales[b] <= 4), and
 * for each such scale the smallest and largest code each element can take.
 * Layout: scales [nb][4] (uint16), qlo/qhi [nb][4][32] (int8), nscales [nb].
 * Returns 0, or -1 if some block admits more than 4 scales (box too wide).
 */
#define NSMAX 4
int orc_q8_0_candidates(const float *h, const float *dh, int64_t K,
                        uint16_t *scales, int8_t *qlo, int8_t *qhi, int32_t *nscales)
{
    int64_t nb = K / QK;
    int rc = 0;
    for (int64_t b = 0; b < nb; b++) {
        const float *x = h + b * QK, *e = dh + b * QK;
        double amax_lo = 0.0, amax_hi = 0.0;
        for (int i = 0; i < QK; i++) {
            double a = fabs((double)x[i]);
            double lo = a - (double)e[i]; if (lo < 0.0) lo = 0.0;
            double hi = a + (double)e[i];
            if (lo > amax_lo) amax_lo = lo;
            if (hi > amax_hi) amax_hi = hi;
        }
        /* fp16 scales reachable from amax in [amax_lo, amax_hi]: the fp32
         * division and the fp16 rounding are monotone, so every value between
         * the two endpoint scales (as consecutive positive fp16 patterns). */
        uint16_t s_lo = orc_f32_to_f16((float)amax_lo / 127.0f);
        uint16_t s_hi = orc_f32_to_f16((float)amax_hi / 127.0f);
        int ns = (int)(s_hi - s_lo) + 1;
        if (ns > NSMAX) { ns = NSMAX; rc = -1; }
        nscales[b] = ns;
        for (int c = 0; c < NSMAX; c++) {
            uint16_t s = (uint16_t)(s_lo + (c < ns ? c : ns - 1));
            scales[b * NSMAX + c] = s;
            float df = orc_f16_to_f32(s);
            for (int i = 0; i < QK; i++) {
                int lo, hi;
                if (df == 0.0f) {
                    lo = hi = 0;
                } else {
                    float id = 1.0f / df;
                    float vlo = ((float)((double)x[i] - (double)e[i])) * id;
                    float vhi = ((float)((double)x[i] + (double)e[i])) * id;
                    lo = (int)roundf(vlo); hi = (int)roundf(vhi);
                    lo = lo > 127 ? 127 : (lo < -127 ? -127 : lo);
                    hi = hi > 127 ? 127 : (hi < -127 ? -127 : hi);
                }
                qlo[(b * NSMAX + c) * QK + i] = (int8_t)lo;
                qhi[(b * NSMAX + c) * QK + i] = (int8_t)hi;
            }
        }
    }
    return rc;
}

/* ------------------------------------------------------------------ */
/* Residual add and RMSNorm between chained MoE layers.                 */
/* ------------------------------------------------------------------ */

/* Pre-norm residual chaining of the Qwen3-series model family (Sec. 2.2);
 * the paper does not spell the norm out, so this is the standard RMSNorm.
 * Per row t of [T][H]:
 *   x_out = x + y   (one binary32 addition; x_out = x when y is NULL)
 *   xn[i] = x_out[i] / sqrt(mean_i x_out[i]^2 + eps) * gamma[i]   in fp64
 * (xn is skipped when NULL). */
void orc_rmsnorm_residual(const float *x, const float *y, const float *gamma, float *x_out,
                          double *xn, int64_t T, int64_t H, double eps)
{
    for (int64_t t = 0; t < T; t++) {
        const float *xr = x + t * H;
        float *vo = x_out + t * H;
        double ss = 0.0;
        for (int64_t i = 0; i < H; i++) {
            const float v = y ? xr[i] + y[t * H + i] : xr[i];
            vo[i] = v;
            ss += (double)v * (double)v;
        }
        if (!xn) continue;
        const double r = 1.0 / sqrt(ss / (double)H + eps);
        for (int64_t i = 0; i < H; i++) xn[t * H + i] = (double)vo[i] * r * (double)gamma[i];
    }
}

/* ------------------------------------------------------------------ */
/* Router top-k (Sec. 2.2: each token goes to its top-k routed experts). */
/* ------------------------------------------------------------------ */

/* Per token t of logits [T][E]: k times, the largest logit not yet taken
 * (scanning in index order and keeping the first of equal values, so equal
 * logits go in increasing index) -> ids[t][j].  Softmax is monotone, so this
 * is the order of the probabilities.  weights[t][j] = the softmax
 * probability of ids[t][j] divided by the sum of the selected
 * probabilities, evaluated in fp64 as exp(l_j - l_max) / sum over the
 * selection of exp(l_i - l_max).  taken: E bytes of scratch. */
void orc_router_topk(const float *logits, int32_t *ids, double *weights, int64_t T, int64_t E,
                     int64_t k, unsigned char *taken)
{
    for (int64_t t = 0; t < T; t++) {
        const float *l = logits + t * E;
        memset(taken, 0, (size_t)E);
        for (int64_t j = 0; j < k; j++) {
            int64_t best = -1;
            for (int64_t e = 0; e < E; e++)
                if (!taken[e] && (best < 0 || l[e] > l[best])) best = e;
            taken[best] = 1;
            ids[t * k + j] = (int32_t)best;
        }
        const double lmax = (double)l[ids[t * k]];
        double sum = 0.0;
        for (int64_t j = 0; j < k; j++) sum += exp((double)l[ids[t * k + j]] - lmax);
        for (int64_t j = 0; j < k; j++)
            weights[t * k + j] = exp((double)l[ids[t * k + j]] - lmax) / sum;
    }
}

/* Threads for the parallel loops above from now on (timing of the oracle on
 * one core and on all of them; the arithmetic does not depend on it). */
void orc_set_threads(int n)
{
    if (n > 0) omp_set_num_threads(n);
}

/* Number of OpenMP threads the parallel loops above use. */
int orc_threads(void)
{
    int n = 1;
    #pragma omp parallel
    {
        #pragma omp single
        n = omp_get_num_threads();
    }
    return n;
}

/* ------------------------------------------------------------------ */
/* The paper's own block format (Sec. 2.3 "Weight quantization": each  */
/* weight an integer in {-7..7} with one FP32 scale per group, two per  */
/* byte; Sec. 3.3: activations quantized per group to 8 bits with an    */
/* FP32 scale, each 4-bit weight held as the unsigned value in {1..15}).*/
/* Readings: 32 per group; weight scale d = amax / 7 and activation     */
/* scale d = amax / 127, each one correctly rounded fp32 division;      */
/* codes round-half-away(v * (1 / d)) clamped to +-7 / +-127; a zero    */
/* scale, or one whose reciprocal overflows fp32, gives zero codes.     */
/* Q4_SYM block, 20 bytes: fp32 d (little endian), then byte j holding  */
/* q_j + 8 in its low and q_{j+16} + 8 in its high nibble.  Q8_F32      */
/* block, 36 bytes: fp32 d, then 32 int8 codes.                         */
/* ------------------------------------------------------------------ */

#define Q4S_BYTES 20
#define Q8F_BYTES 36

static void wrf32(uint8_t *p, float f) { memcpy(p, &f, 4); }
static float rdf32(const uint8_t *p) { float f; memcpy(&f, p, 4); return f; }

/* the fp32 reciprocal of a scale, or 0 when codes are all zero */
static float sym_inverse(float d)
{
    if (d == 0.0f) return 0.0f;
    float id = 1.0f / d;
    return isinf(id) ? 0.0f : id;
}

static int round_clamp(float v, int lim)
{
    int q = (int)roundf(v);                   /* half away from zero */
    if (q > lim) q = lim;
    if (q < -lim) q = -lim;
    return q;
}

void orc_q4_sym_block(const float *w, uint8_t *out)
{
    float amax = 0.0f;
    for (int i = 0; i < QK; i++) {
        float a = fabsf(w[i]);
        if (a > amax) amax = a;
    }
    float d = amax / 7.0f;
    float id = sym_inverse(d);
    int q[QK];
    for (int i = 0; i < QK; i++)
        q[i] = (id == 0.0f) ? 0 : round_clamp(w[i] * id, 7);
    wrf32(out, d);
    for (int j = 0; j < 16; j++)
        out[4 + j] = (uint8_t)((q[j] + 8) | ((q[j + 16] + 8) << 4));
}

void orc_q8_f32_block(const float *x, uint8_t *out)
{
    float amax = 0.0f;
    for (int i = 0; i < QK; i++) {
        float a = fabsf(x[i]);
        if (a > amax) amax = a;
    }
    float d = amax / 127.0f;
    float id = sym_inverse(d);
    wrf32(out, d);
    for (int i = 0; i < QK; i++)
        out[4 + i] = (uint8_t)(int8_t)((id == 0.0f) ? 0 : round_clamp(x[i] * id, 127));
}

void orc_q4_sym_quantize(const float *w, uint8_t *out, int64_t rows, int64_t K)
{
    int64_t nb = K / QK;
    #pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < rows; r++)
        for (int64_t b = 0; b < nb; b++)
            orc_q4_sym_block(w + r * K + b * QK, out + (r * nb + b) * Q4S_BYTES);
}

void orc_q8_f32_quantize(const float *x, uint8_t *out, int64_t rows, int64_t K)
{
    int64_t nb = K / QK;
    #pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < rows; r++)
        for (int64_t b = 0; b < nb; b++)
            orc_q8_f32_block(x + r * K + b * QK, out + (r * nb + b) * Q8F_BYTES);
}

/* s = sum_i (nibble_i - 8) * q_a,i over one block of the paper's format. */
int32_t orc_blockdot_sym(const uint8_t *wb, const uint8_t *ab)
{
    const int8_t *qa = (const int8_t *)(ab + 4);
    int32_t s = 0;
    for (int j = 0; j < 16; j++) {
        int lo = (wb[4 + j] & 0x0F) - 8;
        int hi = (wb[4 + j] >> 4) - 8;
        s += lo * qa[j] + hi * qa[j + 16];
    }
    return s;
}

/* y[n] = sum_b d_w[n,b] * d_a[b] * s[n,b] in fp64, block order; R[n] = sum
 * of |term|.  Either output pointer may be NULL. */
void orc_gemv_sym(const uint8_t *w, const uint8_t *xq, int64_t N, int64_t K,
                  double *y, double *R)
{
    int64_t nb = K / QK;
    #pragma omp parallel for schedule(static)
    for (int64_t n = 0; n < N; n++) {
        double acc = 0.0, mag = 0.0;
        for (int64_t b = 0; b < nb; b++) {
            const uint8_t *wb = w + (n * nb + b) * Q4S_BYTES;
            const uint8_t *ab = xq + b * Q8F_BYTES;
            double t = (double)rdf32(wb) * (double)rdf32(ab) * (double)orc_blockdot_sym(wb, ab);
            acc += t;
            mag += fabs(t);
        }
        if (y) y[n] = acc;
        if (R) R[n] = mag;
    }
}

/* ------------------------------------------------------------------ */
/* The MoE layer in the paper's own format (Sec. 2.2 layer, Sec. 2.3  */
/* weights, Sec. 3.3 activations and product): the steps of orc_moe   */
/* with Q4_SYM weights, Q8_F32 quantization of x (once per token) and */
/* of h (per token-expert pair), and the products of orc_gemv_sym.    */
/* gu/Rgu/h/hq outputs and hq_in (codes of h to use in the down       */
/* product) as in orc_moe; hq blocks are Q8_F32 (36 bytes).           */
/* ------------------------------------------------------------------ */
int orc_moe_sym(const float *hidden, const int32_t *ids, const float *wts,
                const uint8_t *w_gu, const uint8_t *w_d,
                const uint8_t *ws_gu, const uint8_t *ws_d,
                int64_t T, int64_t H, int64_t I, int64_t E, int64_t k,
                const uint8_t *hq_in,
                double *out, double *R,
                float *gu_out, double *Rgu_out, float *h_out, uint8_t *hq_out,
                const double *shared_w)
{
    int64_t nbH = H / QK, nbI = I / QK;
    size_t gu_bytes = (size_t)(2 * I) * nbH * Q4S_BYTES;   /* one expert's gate/up */
    size_t d_bytes = (size_t)H * nbI * Q4S_BYTES;          /* one expert's down    */
    for (int64_t i = 0; i < T * k; i++)
        if (ids[i] >= E) return -1;

    int bad = 0;
    #pragma omp parallel for schedule(dynamic, 1)
    for (int64_t t = 0; t < T; t++) {
        uint8_t *xq = malloc((size_t)nbH * Q8F_BYTES);
        uint8_t *hq = malloc((size_t)nbI * Q8F_BYTES);
        double *gu = malloc(sizeof(double) * 2 * I);
        double *rgu = malloc(sizeof(double) * 2 * I);
        float *h = malloc(sizeof(float) * I);
        double *y = malloc(sizeof(double) * H);
        double *ry = malloc(sizeof(double) * H);
        if (!xq || !hq || !gu || !rgu || !h || !y || !ry) { bad = 1; goto done; }

        orc_q8_f32_quantize(hidden + t * H, xq, 1, H);
        for (int64_t n = 0; n < H; n++) { out[t * H + n] = 0.0; R[t * H + n] = 0.0; }

        for (int64_t j = 0; j <= k; j++) {
            const uint8_t *Wgu, *Wd;
            double wj;
            int64_t pair;
            if (j < k) {
                int32_t e = ids[t * k + j];
                if (e < 0) continue;
                Wgu = w_gu + (size_t)e * gu_bytes;
                Wd = w_d + (size_t)e * d_bytes;
                wj = (double)wts[t * k + j];
                pair = t * k + j;
            } else {
                if (!ws_gu || !ws_d) continue;
                Wgu = ws_gu;
                Wd = ws_d;
                wj = shared_w ? shared_w[t] : 1.0;
                pair = T * k + t;
            }
            orc_gemv_sym(Wgu, xq, 2 * I, H, gu, rgu);
            for (int64_t i = 0; i < I; i++) {
                float g = (float)gu[i], u = (float)gu[I + i];
                h[i] = (float)(silu_d((double)g) * (double)u);
            }
            if (gu_out) for (int64_t i = 0; i < 2 * I; i++) gu_out[pair * 2 * I + i] = (float)gu[i];
            if (Rgu_out) for (int64_t i = 0; i < 2 * I; i++) Rgu_out[pair * 2 * I + i] = rgu[i];
            if (h_out) memcpy(h_out + pair * I, h, sizeof(float) * I);
            orc_q8_f32_quantize(h, hq, 1, I);
            if (hq_out) memcpy(hq_out + pair * nbI * Q8F_BYTES, hq, (size_t)nbI * Q8F_BYTES);
            const uint8_t *hq_use = hq_in ? hq_in + pair * nbI * Q8F_BYTES : hq;
            orc_gemv_sym(Wd, hq_use, H, I, y, ry);
            for (int64_t n = 0; n < H; n++) {
                out[t * H + n] += wj * y[n];
                R[t * H + n] += fabs(wj) * ry[n];
            }
        }
    done:
        free(xq); free(hq); free(gu); free(rgu); free(h); free(y); free(ry);
    }
    return bad ? -2 : 0;
}
