/*
 * EFQ-Softmax CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, deliberately unoptimised implementation of what the GPU
 * path computes, written from the paper "EFQ-Softmax: Exp-Free Quantization
 * for Softmax" (arXiv 2609.09721).  Only the test-suite, the smoke check and
 * the CPU-baseline leg of the benchmark may load this file; the product
 * library never links or calls it, and it shares no code, header, table or
 * constant with the HIP sources.
 *
 * What is computed, and where the paper defines it:
 *   - V -> MXFP4 (orc_quant_v): the "existing low-bit path" for the value
 *     operand, Sec. III-A, Eq. (numerator-lowbit).  The paper does not fix
 *     the rule; this follows the OCP microscaling (MX v1.0) MXFP4 encoding:
 *     shared exponent floor(log2 amax) - 2, E2M1 elements rounded to nearest
 *     (ties to even mantissa), saturating at 6.
 *   - P-gen for one microscaling block (pgen_block): Algorithm 1, i.e.
 *     Eq. (k-rule) for the scale exponent, Eq. (z-def) for the residual and
 *     Eq. (d8-index) for the code (EFQ), or the 16-level index j16 folded by
 *     the table C16 of Sec. II-D (EFQ-Softmax-LUT).
 *   - Exp-then-quantize baseline (pgen_block_expq): Eq. (post-softmax-path):
 *     FP32 probabilities exp(x), then the OCP MXFP4 quantiser, or (ORC_EXPQ6)
 *     the "scale6" exponent ceil(log2(amax / 6)) of the paper's comparison
 *     rows (Sec. IV).
 *   - Low-bit Q K^T (orc_quant_mxfp8, orc_attn with qk8 set): the paper
 *     frames low-bit attention as running Q K^T (and P V) on FP8/FP4 matrix
 *     engines (Sec. I).  Q and K are then MXFP8 under the OCP microscaling
 *     rule: per 32 consecutive elements along head_dim, shared exponent
 *     floor(log2 amax) - 8 (8 = largest E4M3 exponent), E4M3 elements
 *     rounded to nearest (ties to even), saturating at 448.
 *   - The online recurrence (orc_attn): Algorithm 2 for every key/value tile
 *     in ascending order: Eqs. (rowmax-update), (alpha), (numerator-basic),
 *     (denominator-basic) and the final division of Sec. III-A.  Algorithm 3
 *     (the offline (tau, h) search of Sec. III-C) is a loop over this call,
 *     in oracle/__init__.py.
 *
 * Floating point.  The accumulators (A, l) and the exact-softmax reference
 * are fp64.  The decisions that produce integers (scale exponent k_b, code
 * c_t) are taken in fp32, in the operation order of the GPU kernel, so that
 * codes and scales can be compared bit for bit:
 *
 *   S_t  = fl(acc_t * scale)                        score, acc_t = fl(q . k_t)
 *   m    = max(m_prev, max_t S_t)                   Eq. (rowmax-update)
 *   x_t  = fl(S_t - m)                              Eq. (shifted-x)
 *   M_b  = max_{t in b} x_t                         Alg. 1, block maximum
 *   k_b  = floor(fl(fl(M_b + log(2/9)) * (1/log2))) Eq. (k-rule), k_b >= -127
 *   off  = fl(fl(k_b * log2) + fl(log6 + tau))      k_b log2 + log6 + tau
 *   B    = -fl(fl(m + off) * h)
 *   EFQ:  w_t = fma(acc_t, 32 fl(scale*h), fl(32 B + 31.5))
 *             ~ 32 (u_t + 1) - 1/2,  u_t = (x_t - k_b log2 - log6 - tau) h
 *                                        = (z_t - tau) h      Eq. (d8-index)
 *         c_t = floor(min(max(rne(w_t), 0), 255) / 32)
 *   LUT:  w_t = fma(acc_t, 16 fl(scale*h), fl(16 B + 15.5)) ~ 16 (u_t + 1) - 1/2
 *         j16 = floor(min(max(rne(w_t), 0), 255) / 16),  c_t = C16[j16]
 *
 * In exact arithmetic floor(min(max(rne(32 v - 1/2), 0), 255) / 32) is
 * clip(floor(v), 0, 7) for every real v (a half-integer 32 n - 1/2 rounds
 * to the even 32 n, and 32 n + 31.5 only occurs at v = n + 1), so c_t is
 * clip(floor(u_t) + 1, 0, 7) of Eq. (d8-index).  With 16 in place of 32 the
 * same argument gives j16 = clip(floor(u_t) + 1, 0, 15) for the LUT index.  The residual argument is
 * one fused multiply-add of the raw dot product with the row and block
 * terms folded into a bias; in fp32 it can differ from a step-by-step
 * evaluation only within a few ulps of a code threshold.  orc_pgen_real
 * evaluates the same steps in fp64 to pin that.
 *
 * Build: gcc -O2 -std=gnu99 -ffp-contract=off -fno-fast-math -fopenmp
 *        -shared -fPIC efq_oracle.c -lm
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ---- fp32 constants, each the fp32 value nearest the real constant ----- */
static const float F_LN2 = 0.693147180559945309417f;   /* log 2      */
static const float F_INVLN2 = 1.44269504088896340736f; /* 1 / log 2  */
static const float F_LOG2_9 = -1.50407739677627407f;   /* log(2/9)   */
static const float F_LN6 = 1.79175946922805500081f;    /* log 6      */

/* Non-negative E2M1 code set C8 (Sec. II-B): the value of bit pattern c. */
static const double C8[8] = {0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0};

/* EFQ-Softmax-LUT fold table C16 (Sec. II-D). */
static const int C16[16] = {0, 1, 1, 1, 1, 1, 2, 2, 3, 3, 4, 5, 5, 6, 7, 7};

enum { ORC_EFQ = 0, ORC_EXPQ = 1, ORC_EXACT = 2, ORC_LUT = 3, ORC_EXPQ6 = 4 };

#define K_MIN (-127) /* smallest E8M0 exponent; 0x00 encodes 2^-127 */
#define K_MAX 127    /* largest finite E8M0 exponent (0xFE)          */

static float bf16_to_f32(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

static int clampi(int v, int lo, int hi) { return v < lo ? lo : (v > hi ? hi : v); }

/* E2M1 code from w ~ 32 (u + 1) - 1/2: round to nearest (ties to even),
 * saturate to [0, 255], keep the multiple of 32.  -inf and NaN give 0. */
static int code_from_w(float w)
{
    float r = nearbyintf(w); /* default rounding: nearest, ties to even */
    if (!(r > 0.0f))
        return 0;
    if (r > 255.0f)
        r = 255.0f;
    return (int)r / 32;
}

/* LUT index from w ~ 16 (u + 1) - 1/2: round to nearest (ties to even),
 * saturate to [0, 255], keep the multiple of 16.  -inf and NaN give 0. */
static int index_from_w16(float w)
{
    float r = nearbyintf(w);
    if (!(r > 0.0f))
        return 0;
    if (r > 255.0f)
        r = 255.0f;
    return (int)r / 16;
}

/* Nearest E2M1 magnitude code for y >= 0 among C8, ties to the even code
 * (even mantissa bit), values beyond 6 saturate to code 7 (value 6).  A
 * brute-force search over the eight values: round-to-nearest-even with
 * saturation, written without any bit tricks. */
static int e2m1_nearest(double y)
{
    int best = 0;
    double bd = fabs(y - C8[0]);
    for (int c = 1; c < 8; ++c) {
        double d = fabs(y - C8[c]);
        if (d < bd || (d == bd && (c % 2) == 0 && (best % 2) != 0)) {
            best = c;
            bd = d;
        }
    }
    return best;
}

/* floor(log2 a) for a finite a > 0 (exact, via the binary exponent). */
static int floor_log2(double a)
{
    int e;
    double m = frexp(a, &e); /* a = m 2^e, m in [0.5, 1) */
    (void)m;
    return e - 1;
}

/* ------------------------------------------------------------------------
 * Algorithm 1 for one microscaling block, fp32 decision contract.
 *
 * The block's scores are given as raw dot products acc[t] (-inf = masked
 * by the attention mask, Sec. III-D: masks act before P-gen), together with
 * the softmax scale and the running row maximum m, so x_t = fl(S_t - m).
 * Writes codes[t] in 0..7 and returns k_b.
 *
 * Diagnostic (margin != NULL): lowers *margin to the smallest distance, in
 * units of the raw dot product, between an argument of this block's
 * decisions and the nearest value where that decision changes (k_b at
 * integer q, an EFQ code at w = 32 n - 1/2, a LUT index at w = 16 n - 1/2).  It
 * does not change any result; a check that compares against an
 * implementation whose dot products differ in the last bits uses it to
 * tell a legitimate code flip from an error.
 * ---------------------------------------------------------------------- */
static int pgen_block(const float *acc, int n, float scale, float m, float tau,
                      float h, int lut, uint8_t *codes, double *margin)
{
    /* Alg. 1: M_b = max_t x_t (masked keys do not take part). */
    float Mb = -INFINITY;
    for (int t = 0; t < n; ++t) {
        if (acc[t] == -INFINITY)
            continue;
        float S = acc[t] * scale;
        float x = S - m;
        if (x > Mb)
            Mb = x;
    }

    /* Alg. 1: k_b = floor((M_b + log(2/9)) / log 2), Eq. (k-rule); s_b = 2^k_b.
     * A block with no visible key gets the smallest exponent. */
    int k;
    if (Mb == -INFINITY) {
        k = K_MIN;
    } else {
        float a = Mb + F_LOG2_9;
        float q = a * F_INVLN2;
        float fq = floorf(q);
        k = fq < (float)K_MIN ? K_MIN : (fq > (float)K_MAX ? K_MAX : (int)fq);
        if (margin && q > (float)K_MIN - 0.5f) {
            double dq = fabs((double)q - nearbyint((double)q));
            double d = dq / ((double)F_INVLN2 * (double)scale);
            if (d < *margin)
                *margin = d;
        }
    }

    /* Alg. 1: z_t = x_t - k_b log2 - log6 (Eq. z-def), then
     * c_t = clip(floor((z_t - tau) h) + 1, 0, 7) (Eq. d8-index), or for the
     * LUT variant j16 = clip(floor((z_t - tau16) h16) + 1, 0, 15), c_t = C16[j16].
     * (z_t - tau) h is evaluated as acc_t (scale h) - (m + k_b log2 + log6 + tau) h;
     * the floor, the +1 and both clips come from rounding
     * 32 ((z_t - tau) h + 1) - 1/2 (EFQ; 16 (...) - 1/2 for the LUT index) to an
     * integer in [0, 255] (header). */
    float kf = (float)k;
    float klog2 = kf * F_LN2;
    float c0 = F_LN6 + tau;
    float off = klog2 + c0;
    float moff = m + off;
    float bias = -(moff * h);
    float sh = scale * h;
    float sh32 = 32.0f * sh;                  /* exact */
    float bias32 = fmaf(bias, 32.0f, 31.5f);  /* fl(32 B + 31.5) */
    float sh16 = 16.0f * sh;                  /* exact */
    float bias16 = fmaf(bias, 16.0f, 15.5f);  /* fl(16 B + 15.5) */
    for (int t = 0; t < n; ++t) {
        if (acc[t] == -INFINITY) {
            codes[t] = 0;
            continue;
        }
        if (lut) {
            float w = fmaf(acc[t], sh16, bias16);
            codes[t] = (uint8_t)C16[index_from_w16(w)];
            if (margin) {
                double nb = nearbyint(((double)w + 0.5) / 16.0);
                nb = nb < 1.0 ? 1.0 : (nb > 15.0 ? 15.0 : nb);
                double d = fabs((double)w - (16.0 * nb - 0.5)) / (double)sh16;
                if (d < *margin)
                    *margin = d;
            }
        } else {
            float w = fmaf(acc[t], sh32, bias32);
            codes[t] = (uint8_t)code_from_w(w);
            if (margin) {
                double nb = nearbyint(((double)w + 0.5) / 32.0);
                nb = nb < 1.0 ? 1.0 : (nb > 7.0 ? 7.0 : nb);
                double d = fabs((double)w - (32.0 * nb - 0.5)) / (double)sh32;
                if (d < *margin)
                    *margin = d;
            }
        }
    }
    return k;
}

/* Smallest integer k with 6 * 2^k >= a, for a finite a > 0: the "scale6"
 * exponent ceil(log2(a / 6)), by search from below an exact lower bound. */
static int ceil_log2_over6(double a)
{
    int k = floor_log2(a) - 3; /* 6 * 2^k < 2^(k+3) <= a */
    while (6.0 * ldexp(1.0, k) < a)
        ++k;
    return k;
}

/* Exp-then-quantize for one block, Eq. (post-softmax-path): p_t = fl32(e^x_t),
 * then an MXFP4 quantiser with elements rounded to nearest even, saturating.
 * Scale exponent: the OCP rule floor(log2 max p) - 2, or with scale6 the
 * rule ceil(log2(max p / 6)) of the paper's MXFP4-scale6 comparison rows
 * (max p / 2^k in (3, 6], so nothing saturates).  Returns k_b. */
static int pgen_block_expq(const float *acc, int n, float scale, float m, int scale6,
                           uint8_t *codes)
{
    float p[64];
    float amax = 0.0f;
    for (int t = 0; t < n; ++t) {
        if (acc[t] == -INFINITY) {
            p[t] = 0.0f;
            continue;
        }
        float S = acc[t] * scale;
        float x = S - m;
        p[t] = (float)exp((double)x);
        if (p[t] > amax)
            amax = p[t];
    }
    int k = K_MIN;
    if (amax > 0.0f)
        k = clampi(scale6 ? ceil_log2_over6((double)amax) : floor_log2((double)amax) - 2,
                   K_MIN, K_MAX);
    for (int t = 0; t < n; ++t)
        codes[t] = (uint8_t)e2m1_nearest(ldexp((double)p[t], -k));
    return k;
}

/* ---------------------------------------------------------------------- *
 * Standalone P-gen unit (Sec. III-D kernel interface): shifted scores x
 * (rows x cols, row-major, -inf = masked) -> codes (one per byte) and one
 * E8M0 byte (k_b + 127) per 32-column block.  The last block of a row may
 * be partial (cols not a multiple of 32).  mode: ORC_EFQ, ORC_LUT, ORC_EXPQ,
 * ORC_EXPQ6.
 * Here x is the score itself: scale 1 and row maximum 0.
 * ---------------------------------------------------------------------- */
int orc_pgen(const float *x, long rows, int cols, int mode, float tau, float h,
             uint8_t *codes, uint8_t *e8m0)
{
    if (!x || !codes || !e8m0 || rows < 0 || cols < 0)
        return -1;
    int nblk = (cols + 31) / 32;
    for (long r = 0; r < rows; ++r) {
        for (int b = 0; b < nblk; ++b) {
            int t0 = b * 32;
            int n = cols - t0 < 32 ? cols - t0 : 32;
            const float *xb = x + r * (long)cols + t0;
            uint8_t *cb = codes + r * (long)cols + t0;
            int k;
            if (mode == ORC_EXPQ || mode == ORC_EXPQ6)
                k = pgen_block_expq(xb, n, 1.0f, 0.0f, mode == ORC_EXPQ6, cb);
            else
                k = pgen_block(xb, n, 1.0f, 0.0f, tau, h, mode == ORC_LUT, cb, NULL);
            e8m0[r * nblk + b] = (uint8_t)(k + 127);
        }
    }
    return 0;
}

/* The same steps in fp64 (real-valued reading of Alg. 1, step by step as
 * printed): M_b, k_b = floor((M_b + log(2/9))/log 2), z_t = x_t - k_b log 2
 * - log 6, c_t = clip(floor((z_t - tau) h) + 1, 0, 7).  Used only to pin the
 * fp32 contract against the paper's formulas.  Also returns u_t. */
int orc_pgen_real(const double *x, long rows, int cols, int lut, double tau, double h,
                  uint8_t *codes, int16_t *kexp, double *u_out)
{
    int nblk = (cols + 31) / 32;
    for (long r = 0; r < rows; ++r) {
        for (int b = 0; b < nblk; ++b) {
            int t0 = b * 32;
            int n = cols - t0 < 32 ? cols - t0 : 32;
            const double *xb = x + r * (long)cols + t0;
            double Mb = -INFINITY;
            for (int t = 0; t < n; ++t)
                if (xb[t] > Mb)
                    Mb = xb[t];
            int k;
            if (Mb == -INFINITY)
                k = K_MIN;
            else
                k = clampi((int)floor((Mb + log(2.0 / 9.0)) / log(2.0)), K_MIN, K_MAX);
            kexp[r * nblk + b] = (int16_t)k;
            for (int t = 0; t < n; ++t) {
                long i = r * (long)cols + t0 + t;
                if (xb[t] == -INFINITY) {
                    codes[i] = 0;
                    u_out[i] = -INFINITY;
                    continue;
                }
                double z = xb[t] - k * log(2.0) - log(6.0);
                double u;
                int c;
                if (lut) {
                    double tau16 = log(1.0 / 24.0), h16 = 14.0 / log(24.0);
                    u = (z - tau16) * h16;
                    double fu = floor(u);
                    int j = fu < -1.0 ? 0 : (fu >= 15.0 ? 15 : (int)fu + 1);
                    c = C16[j];
                } else {
                    u = (z - tau) * h;
                    double fu = floor(u);
                    c = fu < -1.0 ? 0 : (fu >= 7.0 ? 7 : (int)fu + 1);
                }
                codes[i] = (uint8_t)c;
                u_out[i] = u;
            }
        }
    }
    return 0;
}

/* ---------------------------------------------------------------------- *
 * V -> MXFP4 along the key dimension.  v: [B][S][H][D] bf16 bits.
 * codes: [B][H][nblk*32][D], one E2M1 code per byte (bit 3 = sign of the
 * bf16 input, keys past S get code 0).  e8m0: [B][H][nblk][D].
 * ---------------------------------------------------------------------- */
int orc_quant_v(const uint16_t *v, int B, int S, int H, int D, uint8_t *codes,
                uint8_t *e8m0)
{
    if (!v || !codes || !e8m0 || B < 0 || S < 0 || H < 0 || D < 0)
        return -1;
    int nblk = (S + 31) / 32;
    for (int b = 0; b < B; ++b)
        for (int g = 0; g < H; ++g)
            for (int blk = 0; blk < nblk; ++blk)
                for (int d = 0; d < D; ++d) {
                    double amax = 0.0;
                    for (int t = blk * 32; t < blk * 32 + 32 && t < S; ++t) {
                        double a = fabs((double)bf16_to_f32(v[(((long)b * S + t) * H + g) * D + d]));
                        if (a > amax)
                            amax = a;
                    }
                    int k = K_MIN;
                    if (amax > 0.0)
                        k = clampi(floor_log2(amax) - 2, K_MIN, K_MAX);
                    e8m0[(((long)b * H + g) * nblk + blk) * D + d] = (uint8_t)(k + 127);
                    for (int t = blk * 32; t < blk * 32 + 32; ++t) {
                        uint8_t c = 0;
                        if (t < S) {
                            uint16_t bits = v[(((long)b * S + t) * H + g) * D + d];
                            double y = fabs((double)bf16_to_f32(bits));
                            c = (uint8_t)e2m1_nearest(ldexp(y, -k));
                            if (bits & 0x8000u)
                                c |= 8u;
                        }
                        codes[(((long)b * H + g) * (long)nblk * 32 + t) * D + d] = c;
                    }
                }
    return 0;
}

/* value of an E2M1 code (bit 3 = sign) times 2^k */
static double e2m1_value(uint8_t c, int k)
{
    double v = ldexp(C8[c & 7u], k);
    return (c & 8u) ? -v : v;
}

/* Magnitude of the E4M3 code c (0 <= c < 0x7F, sign bit clear): exponent
 * field e (bias 7), mantissa m; e = 0 is subnormal, m * 2^-9.  0x7F is NaN
 * and is never produced. */
static double e4m3_magnitude(int c)
{
    int e = (c >> 3) & 15, m = c & 7;
    return e == 0 ? ldexp((double)m, -9) : ldexp(1.0 + m / 8.0, e - 7);
}

/* Nearest E4M3 magnitude code for y >= 0, ties to the even code (even
 * mantissa bit), values above 448 saturate to 448 (code 0x7E).  The 127
 * finite non-negative codes increase with their magnitude: bisect for the
 * last code c whose magnitude is <= y, then take c or c + 1, whichever is
 * nearer. */
static int e4m3_nearest(double y)
{
    if (y >= e4m3_magnitude(0x7E))
        return 0x7E;
    int lo = 0, hi = 0x7E; /* magnitude(lo) <= y < magnitude(hi) */
    while (hi - lo > 1) {
        int mid = (lo + hi) / 2;
        if (e4m3_magnitude(mid) <= y)
            lo = mid;
        else
            hi = mid;
    }
    double dl = y - e4m3_magnitude(lo), dh = e4m3_magnitude(hi) - y;
    if (dl < dh)
        return lo;
    if (dh < dl)
        return hi;
    return (lo % 2 == 0) ? lo : hi;
}

/* ------------------------------------------------------------------------
 * MXFP8 (E4M3) quantiser for Q and K: x is rows x D bf16 bits (D a multiple
 * of 32); for each row and 32-element block: k = floor(log2 amax) - 8
 * clamped to [-127, 127] (amax = 0: k = -127), codes = sign | nearest
 * E4M3 of |x| 2^-k.  codes: rows x D bytes, e8m0: rows x D/32 bytes (k+127).
 * ---------------------------------------------------------------------- */
int orc_quant_mxfp8(const uint16_t *x, long rows, int D, uint8_t *codes, uint8_t *e8m0)
{
    if (!x || !codes || !e8m0 || rows < 0 || D < 32 || D % 32 != 0)
        return -1;
    for (long r = 0; r < rows; ++r)
        for (int blk = 0; blk < D / 32; ++blk) {
            const uint16_t *xb = x + r * D + blk * 32;
            double amax = 0.0;
            for (int t = 0; t < 32; ++t) {
                double a = fabs((double)bf16_to_f32(xb[t]));
                if (a > amax)
                    amax = a;
            }
            int k = K_MIN;
            if (amax > 0.0)
                k = clampi(floor_log2(amax) - 8, K_MIN, K_MAX);
            e8m0[r * (D / 32) + blk] = (uint8_t)(k + 127);
            for (int t = 0; t < 32; ++t) {
                double y = fabs((double)bf16_to_f32(xb[t]));
                int c = e4m3_nearest(ldexp(y, -k));
                if (xb[t] & 0x8000u)
                    c |= 0x80;
                codes[r * D + blk * 32 + t] = (uint8_t)c;
            }
        }
    return 0;
}

/* value of an MXFP8 element: E4M3 code (bit 7 = sign) times 2^k */
static double e4m3_value(uint8_t c, int k)
{
    double v = ldexp(e4m3_magnitude(c & 0x7F), k);
    return (c & 0x80u) ? -v : v;
}

/* Q or K as the values the low-bit Q K^T multiplies: [rows][D] doubles. */
static double *mxfp8_values(const uint16_t *x, long rows, int D)
{
    uint8_t *c = malloc((size_t)rows * D);
    uint8_t *e = malloc((size_t)rows * (D / 32));
    double *out = malloc(sizeof(double) * (size_t)rows * D);
    if (!c || !e || !out || orc_quant_mxfp8(x, rows, D, c, e) != 0) {
        free(c);
        free(e);
        free(out);
        return NULL;
    }
    for (long r = 0; r < rows; ++r)
        for (int d = 0; d < D; ++d)
            out[r * D + d] = e4m3_value(c[r * D + d], (int)e[r * (D / 32) + d / 32] - 127);
    free(c);
    free(e);
    return out;
}

/* ---------------------------------------------------------------------- *
 * Attention forward for a list of query rows, Algorithm 2 over key/value
 * tiles of width bc (a multiple of 32) in ascending key order.
 *
 * q: [B][Sq][Hq][D], k, v: [B][Sk][Hkv][D] (bf16 bits).  GQA: query head hq
 * reads key/value head hq / (Hq/Hkv).  causal (requires Sq == Sk): key t is
 * visible to query i iff t <= i.  Keys t >= Sk are padding (masked).
 * rows: nrows triples (b, hq, i).  out: [nrows][D] fp32.
 * mode ORC_EFQ / ORC_LUT: P from Alg. 1, V as MXFP4.  ORC_EXPQ (ORC_EXPQ6,
 * scale6 rule): P from the
 * exp-then-quantize path, V as MXFP4.  ORC_EXACT: fp64 softmax with
 * unquantised V (the unquantised reference of the calibration objective).
 * Optional dumps (may be NULL): codes [nrows][nblk*32] (one code per byte),
 * e8m0 [nrows][nblk], final m (fp32, score units) and l (fp64) per row,
 * and row_margin [nrows]: the smallest decision margin of the row (EFQ and
 * LUT; see pgen_block), +inf when no decision was taken.
 * ---------------------------------------------------------------------- */
int orc_attn(const uint16_t *q, const uint16_t *kmat, const uint16_t *v, int B, int Sq,
             int Sk, int Hq, int Hkv, int D, float scale, int causal, int mode, float tau,
             float h, int bc, const int32_t *rows, long nrows, float *out,
             uint8_t *dump_codes, uint8_t *dump_e8m0, float *dump_m, double *dump_l,
             double *row_margin, int qk8, int nthreads)
{
    if (!q || !kmat || !v || !rows || !out || B < 1 || Sq < 1 || Sk < 1 || Hq < 1 ||
        Hkv < 1 || D < 1 || Hq % Hkv != 0 || bc < 32 || bc % 32 != 0 || bc > 1024)
        return -1;
    if (causal && Sq != Sk)
        return -1;
    const int nblk = (Sk + 31) / 32;
    const int group = Hq / Hkv;
    const int quant = (mode != ORC_EXACT);
    if (qk8 && D % 32 != 0)
        return -1;
    /* low-bit Q K^T: K as its MXFP8 values (each Q row is quantised when
     * its row is processed) */
    double *k8 = NULL;
    if (qk8) {
        k8 = mxfp8_values(kmat, (long)B * Sk * Hkv, D);
        if (!k8)
            return -2;
    }

    /* Quantised V for every (b, kv head): [B][Hkv][nblk*32][D] values. */
    double *vhat = NULL;
    if (quant) {
        uint8_t *vc = malloc((size_t)B * Hkv * nblk * 32 * D);
        uint8_t *ve = malloc((size_t)B * Hkv * nblk * D);
        vhat = malloc(sizeof(double) * (size_t)B * Hkv * nblk * 32 * D);
        if (!vc || !ve || !vhat) {
            free(vc);
            free(ve);
            free(vhat);
            return -2;
        }
        orc_quant_v(v, B, Sk, Hkv, D, vc, ve);
        for (long b = 0; b < B; ++b)
            for (long g = 0; g < Hkv; ++g)
                for (long t = 0; t < (long)nblk * 32; ++t)
                    for (long d = 0; d < D; ++d) {
                        long ci = ((b * Hkv + g) * nblk * 32 + t) * D + d;
                        int kv = (int)ve[((b * Hkv + g) * nblk + t / 32) * D + d] - 127;
                        vhat[ci] = e2m1_value(vc[ci], kv);
                    }
        free(vc);
        free(ve);
    }

#ifdef _OPENMP
    if (nthreads > 0)
        omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
    int fail = 0;
#pragma omp parallel for schedule(dynamic, 1)
    for (long r = 0; r < nrows; ++r) {
        const int b = rows[3 * r], hq = rows[3 * r + 1], i = rows[3 * r + 2];
        if (b < 0 || b >= B || hq < 0 || hq >= Hq || i < 0 || i >= Sq) {
            fail = 1;
            continue;
        }
        const int g = hq / group;
        float *acc = malloc(sizeof(float) * bc);
        uint8_t *cd = malloc((size_t)bc);
        double *A = calloc((size_t)D, sizeof(double));
        double *dA = calloc((size_t)D, sizeof(double));
        double *qd = malloc(sizeof(double) * D);
        if (!acc || !cd || !A || !dA || !qd) {
            fail = 1;
            free(acc); free(cd); free(A); free(dA); free(qd);
            continue;
        }
        const long q0 = (((long)b * Sq + i) * Hq + hq) * D;
        double *qrow8 = qk8 ? mxfp8_values(q + q0, 1, D) : NULL;
        if (qk8 && !qrow8) {
            fail = 1;
            free(acc); free(cd); free(A); free(dA); free(qd);
            continue;
        }
        for (int d = 0; d < D; ++d)
            qd[d] = qk8 ? qrow8[d] : (double)bf16_to_f32(q[q0 + d]);
        free(qrow8);
        /* blocks that are never processed (past the causal limit) read as
         * fully masked blocks: codes 0 and E8M0 0x00 */
        if (dump_codes)
            memset(dump_codes + r * (long)nblk * 32, 0, (size_t)nblk * 32);
        if (dump_e8m0)
            memset(dump_e8m0 + r * (long)nblk, 0, (size_t)nblk);
        const int kend = causal ? i + 1 : Sk; /* keys [0, kend) are visible */
        double margin = INFINITY;             /* diagnostic, see pgen_block */
        float m = -INFINITY;                  /* running max, score units */
        double mx = -INFINITY;                /* running max, fp64 (EXACT) */
        double l = 0.0;

        for (int j0 = 0; j0 < Sk; j0 += bc) {
            if (j0 >= kend)
                break; /* fully masked tile: exact no-op (alpha = 1, no terms) */
            const int nt = Sk - j0 < bc ? Sk - j0 : bc;
            /* Alg. 2: S = Q K^T / sqrt(d) (+ mask); acc_t = fl32 of the fp64 dot. */
            double dots[1024];
            for (int t = 0; t < bc; ++t) {
                int key = j0 + t;
                if (t >= nt || key >= kend) {
                    acc[t] = -INFINITY;
                    dots[t] = -INFINITY;
                    continue;
                }
                const long kb0 = (((long)b * Sk + key) * Hkv + g) * D;
                double s = 0.0;
                for (int d = 0; d < D; ++d)
                    s += qd[d] * (qk8 ? k8[kb0 + d] : (double)bf16_to_f32(kmat[kb0 + d]));
                acc[t] = (float)s;
                dots[t] = s;
            }
            for (int d = 0; d < D; ++d)
                dA[d] = 0.0;
            double dl = 0.0;

            if (mode == ORC_EXACT) {
                /* exact online softmax in fp64, Eqs. (rowmax-update)-(exact-l) */
                double mt = mx;
                for (int t = 0; t < nt; ++t)
                    if (dots[t] != -INFINITY && dots[t] * scale > mt)
                        mt = dots[t] * scale;
                double alpha = (mx == -INFINITY) ? 0.0 : exp(mx - mt);
                for (int t = 0; t < nt; ++t) {
                    if (dots[t] == -INFINITY)
                        continue;
                    double p = exp(dots[t] * scale - mt);
                    const uint16_t *vr = v + (((long)b * Sk + j0 + t) * Hkv + g) * D;
                    for (int d = 0; d < D; ++d)
                        dA[d] += p * (double)bf16_to_f32(vr[d]);
                    dl += p;
                }
                for (int d = 0; d < D; ++d)
                    A[d] = alpha * A[d] + dA[d];
                l = alpha * l + dl;
                mx = mt;
                continue;
            }

            /* Alg. 2: m^j = max(m^{j-1}, rowmax S^j), Eq. (rowmax-update). */
            float mnew = m;
            for (int t = 0; t < nt; ++t) {
                if (acc[t] == -INFINITY)
                    continue;
                float S = acc[t] * scale;
                if (S > mnew)
                    mnew = S;
            }
            /* Alg. 2: alpha = exp(m^{j-1} - m^j), Eq. (alpha). */
            double alpha = (m == -INFINITY) ? 0.0 : exp((double)m - (double)mnew);

            /* Alg. 2: P-gen per microscaling block (Alg. 1), then
             * dA = P~ V (Eq. numerator-basic) and dl = P~ 1 (Eq.
             * denominator-basic) from the same operand. */
            for (int b0 = 0; b0 < bc; b0 += 32) {
                int kb;
                if (mode == ORC_EXPQ || mode == ORC_EXPQ6)
                    kb = pgen_block_expq(acc + b0, 32, scale, mnew, mode == ORC_EXPQ6, cd + b0);
                else
                    kb = pgen_block(acc + b0, 32, scale, mnew, tau, h, mode == ORC_LUT,
                                    cd + b0, row_margin ? &margin : NULL);
                int blk = (j0 + b0) / 32;
                if (blk < nblk) {
                    if (dump_e8m0)
                        dump_e8m0[r * nblk + blk] = (uint8_t)(kb + 127);
                    if (dump_codes)
                        memcpy(dump_codes + r * (long)nblk * 32 + (long)blk * 32, cd + b0, 32);
                }
                for (int t = b0; t < b0 + 32 && t < nt; ++t) {
                    if (cd[t] == 0)
                        continue;
                    double p = ldexp(C8[cd[t]], kb);
                    const double *vr = vhat + (((long)b * Hkv + g) * nblk * 32 + j0 + t) * D;
                    for (int d = 0; d < D; ++d)
                        dA[d] += p * vr[d];
                    dl += p;
                }
            }
            /* Alg. 2: A = alpha A + dA, l = alpha l + dl. */
            for (int d = 0; d < D; ++d)
                A[d] = alpha * A[d] + dA[d];
            l = alpha * l + dl;
            m = mnew;
        }
        /* Final normalisation O = A / l (Sec. III-A). */
        for (int d = 0; d < D; ++d)
            out[r * D + d] = (l > 0.0) ? (float)(A[d] / l) : 0.0f;
        if (dump_m)
            dump_m[r] = (mode == ORC_EXACT) ? (float)mx : m;
        if (dump_l)
            dump_l[r] = l;
        if (row_margin)
            row_margin[r] = margin;
        free(acc); free(cd); free(A); free(dA); free(qd);
    }
    free(vhat);
    free(k8);
    return fail ? -1 : 0;
}

/* Version tag so the Python side can tell a stale build. */
int orc_version(void) { return 3; }
