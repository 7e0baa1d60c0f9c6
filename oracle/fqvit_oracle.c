/*
 * fqvit_oracle.c -- plain, slow, scalar CPU oracle for FQ-ViT's integer hot path.
 *
 * TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the CPU
 * baseline leg of the benchmark load this library; the HIP library never
 * does and shares no code with it.
 *
 * Each function takes the paper's steps in the paper's order and notation:
 *   Sec. 3.1, eq. (3)-(5)    uniform MinMax quantizer
 *   Sec. 3.2, eq. (8)-(12)   PTF quantizer, its argmin for alpha, phase-1 shift
 *   Supplement A.1           integer LayerNorm: M1, M2, the sqrt approximation,
 *                            A, B, the dyadic N1/N2 form and the output Y_Q
 *   Supplement A.2, Alg. 1   I-Exp
 *   Supplement A.2, Alg. 2   I-Log2 and Log-Int-Softmax, with the clip of the
 *                            LIS equation in the same section
 *   Sec. 3.3 eq. (16)-(17)   BitShift Attn x V; the zero-point form of the same
 *   and Supplement A.2       product in the supplement
 *
 * Integers are exact (int64, or unsigned __int128 where a sum could be wide).
 * Real-valued quantities that the paper leaves as reals are IEEE double with
 * every operation rounded separately (build with -ffp-contract=off).
 * Choices the paper does not fix are marked READING.
 *
 * Build: gcc -std=gnu11 -O2 -ffp-contract=off -fno-fast-math -fPIC -shared
 */
#include "fqvit_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------ */
/* small exact helpers                                                       */
/* ------------------------------------------------------------------------ */

/* floor(a / b) for integers of any sign, b != 0. */
static int64_t floor_div(int64_t a, int64_t b) {
    int64_t q = a / b;
    int64_t r = a % b;
    if (r != 0 && ((r < 0) != (b < 0))) q -= 1;
    return q;
}

static int64_t clip_i64(int64_t x, int64_t lo, int64_t hi) {
    return x < lo ? lo : (x > hi ? hi : x);
}

static double clip_d(double x, double lo, double hi) {
    return x < lo ? lo : (x > hi ? hi : x);
}

/* The paper's rounding bracket.  READING: ties are not specified; the oracle
 * uses round-half-to-even, which is what nearbyint() does in the default
 * rounding mode. */
static double round_nearest(double x) { return nearbyint(x); }

/* ------------------------------------------------------------------------ */
/* Sec. 3.1, eq. (3)-(5): uniform MinMax quantizer                           */
/* ------------------------------------------------------------------------ */

int oracle_minmax_params(const double* x, int64_t n, int32_t b, double* s, int32_t* zp) {
    if (!x || !s || !zp || n <= 0 || b < 1 || b > 16) return ORACLE_ERR_ARG;
    double l = x[0], u = x[0];                        /* eq. (4) */
    for (int64_t i = 1; i < n; ++i) {
        if (x[i] < l) l = x[i];
        if (x[i] > u) u = x[i];
    }
    const double levels = (double)((1 << b) - 1);
    *s = (u - l) / levels;                            /* eq. (5) */
    if (!(*s > 0.0)) return ORACLE_ERR_ARG;
    *zp = (int32_t)clip_d(round_nearest(-l / *s), 0.0, levels);
    return ORACLE_OK;
}

int oracle_minmax_quantize(const double* x, int64_t n, double s, int32_t zp, int32_t b,
                           int32_t* q) {
    if (!x || !q || n < 0 || b < 1 || b > 16 || !(s > 0.0)) return ORACLE_ERR_ARG;
    const double levels = (double)((1 << b) - 1);
    for (int64_t i = 0; i < n; ++i)                   /* eq. (3) */
        q[i] = (int32_t)clip_d(round_nearest(x[i] / s) + (double)zp, 0.0, levels);
    return ORACLE_OK;
}

/* ------------------------------------------------------------------------ */
/* Sec. 3.2, eq. (8)-(11): Power-of-Two-Factor quantizer                      */
/* ------------------------------------------------------------------------ */

int oracle_ptf_params(const double* x, int64_t T, int32_t C, int32_t b, int32_t K,
                      double* s, int32_t* zp) {
    if (!x || !s || !zp || T <= 0 || C <= 0 || b < 1 || b > 16 || K < 0 || K > 30)
        return ORACLE_ERR_ARG;
    const int64_t n = T * (int64_t)C;
    double mn = x[0], mx = x[0];
    for (int64_t i = 1; i < n; ++i) {
        if (x[i] < mn) mn = x[i];
        if (x[i] > mx) mx = x[i];
    }
    const double levels = (double)((1 << b) - 1);
    const double two_K = ldexp(1.0, K);
    *s = (mx - mn) / levels / two_K;                  /* eq. (9)  */
    if (!(*s > 0.0)) return ORACLE_ERR_ARG;
    *zp = (int32_t)clip_d(round_nearest(-mn / (two_K * *s)), 0.0, levels);   /* eq. (10) */
    return ORACLE_OK;
}

/* eq. (8) for one value on the unsigned grid. */
static double ptf_q(double x, double s, int32_t zp, int32_t alpha, double levels) {
    return clip_d(round_nearest(x / (ldexp(1.0, alpha) * s)) + (double)zp, 0.0, levels);
}

/* ---- exact sums of binary64 values --------------------------------------
 * An exact accumulator: a signed fixed-point integer with 32-bit digits whose
 * least significant bit is 2^-1127, below the least significant bit of any
 * binary64 significand (subnormals included), and whose top digit reaches
 * past 2^1024.  Each added double m 2^e (m a 53-bit integer) lands in three
 * consecutive digits; the digits are int64, so up to 2^31 additions fit
 * before any carry is propagated.  The value is the exact sum of everything
 * added, independent of the order of the additions. */
#define XACC_LSB_EXP (-1127)
#define XACC_DIGITS 72

typedef struct {
    int64_t d[XACC_DIGITS];
} xacc;

static void xacc_add(xacc* acc, double v) {
    if (v == 0.0) return;
    int e = 0;
    const double f = frexp(fabs(v), &e);            /* |v| = f 2^e, f in [0.5, 1) */
    const uint64_t m = (uint64_t)ldexp(f, 53);      /* |v| = m 2^(e - 53), exact    */
    const int pos = e - 53 - XACC_LSB_EXP;          /* bit index of m's lowest bit  */
    const int di = pos / 32, sh = pos % 32;
    const unsigned __int128 w = (unsigned __int128)m << sh;   /* below 2^85 */
    const int64_t sgn = v < 0.0 ? -1 : 1;
    for (int k = 0; k < 3 && di + k < XACC_DIGITS; ++k)
        acc->d[di + k] += sgn * (int64_t)(uint32_t)(w >> (32 * k));
}

/* Carry propagation: every digit but the top one in [0, 2^32). */
static void xacc_normalize(xacc* acc) {
    for (int i = 0; i + 1 < XACC_DIGITS; ++i) {
        const int64_t carry = acc->d[i] >> 32;      /* floor division by 2^32 */
        acc->d[i] -= carry * ((int64_t)1 << 32);
        acc->d[i + 1] += carry;
    }
}

/* Sign of a - b (-1, 0, 1), exactly. */
static int xacc_cmp(const xacc* a, const xacc* b) {
    xacc t;
    for (int i = 0; i < XACC_DIGITS; ++i) t.d[i] = a->d[i] - b->d[i];
    xacc_normalize(&t);
    for (int i = XACC_DIGITS - 1; i >= 0; --i)
        if (t.d[i] != 0) return (i == XACC_DIGITS - 1 && t.d[i] < 0) ? -1 : 1;
    return 0;
}

/* The accumulated value rounded to a double (the three top digits summed in
 * long double, then rounded: within one unit in the last place).  acc must
 * be normalized. */
static double xacc_value(const xacc* acc) {
    if (acc->d[XACC_DIGITS - 1] < 0) {            /* negative: the value of -acc, negated */
        xacc neg;
        for (int i = 0; i < XACC_DIGITS; ++i) neg.d[i] = -acc->d[i];
        xacc_normalize(&neg);
        return -xacc_value(&neg);
    }
    int top = XACC_DIGITS - 1;
    while (top > 0 && acc->d[top] == 0) --top;
    long double v = 0.0L;
    for (int i = top; i >= 0 && i >= top - 2; --i)
        v += ldexpl((long double)acc->d[i], 32 * i + XACC_LSB_EXP);
    return (double)v;
}

/* The accumulated value as an unevaluated pair hi + lo: hi as xacc_value,
 * lo the rest of the exact value, rounded.  acc must be normalized. */
static void xacc_value2(const xacc* acc, double* hi, double* lo) {
    *hi = xacc_value(acc);
    xacc rest = *acc;
    xacc_add(&rest, -*hi);
    xacc_normalize(&rest);
    *lo = xacc_value(&rest);
}

/* Error-free product: hi + lo = a b exactly (no underflow assumed). */
static void two_prod(double a, double b, double* hi, double* lo) {
    *hi = a * b;
    *lo = fma(a, b, -*hi);
}

/* Error-free sum: hi + lo = a + b exactly. */
static void two_sum(double a, double b, double* hi, double* lo) {
    *hi = a + b;
    const double bb = *hi - a;
    *lo = (a - (*hi - bb)) + (b - bb);
}

/* Adds (x - k step)^2 to acc exactly.  With k step = p + p' and
 * x - p = u + u' (error-free), the difference is u + u' - p' and its square
 * is the sum of the six exact products of those three terms. */
static void add_exact_sq_err(xacc* acc, double x, double k, double step) {
    double p, pl, u, ul;
    two_prod(k, step, &p, &pl);
    two_sum(x, -p, &u, &ul);
    const double t[3] = {u, ul, -pl};
    for (int i = 0; i < 3; ++i)
        for (int j = i; j < 3; ++j) {
            double h, l;
            two_prod(t[i], t[j], &h, &l);
            const double f = (i == j) ? 1.0 : 2.0;
            xacc_add(acc, f * h);
            xacc_add(acc, f * l);
        }
}

/* eq. (11) for every channel and candidate: err[c (K+1) + a] (+ err_lo[...]
 * when err_lo is non-null) receives the exact error sum_t (x_tc - deq_a(x_tc))^2
 * as an unevaluated pair (see xacc_value2) and,
 * when alpha is non-null, alpha[c] the argmin over a (exact comparison, ties to
 * the smallest a).  deq_a is the quantizer of eq. (8) on the grid 2^a s with its
 * zero point and clip, dequantized: (clip(round(x / (2^a s)) + zp) - zp) 2^a s,
 * the quotient rounded in binary64 as in oracle_ptf_quantize.
 * READING: the printed argmin omits zp and the clip; taken literally the finest
 * grid always wins.  The error is measured on the quantizer that is actually
 * used.  READING: the norm is computed exactly (the exact square of the exact
 * difference, summed exactly), so the result does not depend on any
 * summation order.  Exactness needs every |x| and s within [2^-300, 2^300]
 * (no underflow in the error-free products); the activations of a network are. */
static int ptf_alpha_impl(const double* x, int64_t T, int32_t C, double s, int32_t zp, int32_t b,
                          int32_t K, uint8_t* alpha, double* err, double* err_lo) {
    if (!x || T <= 0 || C <= 0 || b < 1 || b > 16 || K < 0 || K > 7 || !(s > 0.0))
        return ORACLE_ERR_ARG;
    if (T > ((int64_t)1 << 26)) return ORACLE_ERR_ARG;     /* 12 T additions per digit < 2^31 */
    const double levels = (double)((1 << b) - 1);
    xacc* acc = (xacc*)malloc(sizeof(xacc) * (size_t)(K + 1));
    if (!acc) return ORACLE_ERR_ARG;
    for (int32_t c = 0; c < C; ++c) {
        memset(acc, 0, sizeof(xacc) * (size_t)(K + 1));
        for (int32_t a = 0; a <= K; ++a) {
            const double step = ldexp(s, a);
            for (int64_t t = 0; t < T; ++t) {
                const double xv = x[t * C + c];
                add_exact_sq_err(&acc[a], xv, ptf_q(xv, s, zp, a, levels) - (double)zp, step);
            }
            xacc_normalize(&acc[a]);
            if (err) {
                double hi, lo;
                xacc_value2(&acc[a], &hi, &lo);
                err[(int64_t)c * (K + 1) + a] = hi;
                if (err_lo) err_lo[(int64_t)c * (K + 1) + a] = lo;
            }
        }
        int32_t best = 0;
        for (int32_t a = 1; a <= K; ++a)
            if (xacc_cmp(&acc[a], &acc[best]) < 0) best = a;
        if (alpha) alpha[c] = (uint8_t)best;
    }
    free(acc);
    return ORACLE_OK;
}

int oracle_ptf_alpha(const double* x, int64_t T, int32_t C, double s, int32_t zp, int32_t b,
                     int32_t K, uint8_t* alpha) {
    if (!alpha) return ORACLE_ERR_ARG;
    return ptf_alpha_impl(x, T, C, s, zp, b, K, alpha, NULL, NULL);
}

int oracle_ptf_alpha_errors(const double* x, int64_t T, int32_t C, double s, int32_t zp,
                            int32_t b, int32_t K, double* err, double* err_lo) {
    if (!err) return ORACLE_ERR_ARG;
    return ptf_alpha_impl(x, T, C, s, zp, b, K, NULL, err, err_lo);
}

int oracle_ptf_quantize(const double* x, int64_t T, int32_t C, double s, int32_t zp,
                        const uint8_t* alpha, int32_t b, int32_t* q) {
    if (!x || !alpha || !q || T < 0 || C <= 0 || b < 1 || b > 16 || !(s > 0.0))
        return ORACLE_ERR_ARG;
    const double levels = (double)((1 << b) - 1);
    for (int64_t t = 0; t < T; ++t)
        for (int32_t c = 0; c < C; ++c)
            q[t * C + c] = (int32_t)ptf_q(x[t * C + c], s, zp, alpha[c], levels);
    return ORACLE_OK;
}

/* ------------------------------------------------------------------------ */
/* Dyadic requantization of an int32 accumulator to a b-bit activation        */
/* ------------------------------------------------------------------------ */

/* The integer-only requantization of the LayerNorm output in Supplement A.1
 * (a real multiplier replaced by N2 / 2^N1, then a rounding shift), applied
 * to an accumulator of scale s_in, e.g. the BitShift product of Sec. 3.3
 * (scale s_V / 2^N), to give the next layer's b-bit input of scale s_out.
 * READING: the precision of N2 for this step is not given; N2 keeps 31
 * significant bits of M = s_in / s_out, i.e.
 *   N1 = clamp(31 - e, 0, 62) with M = f 2^e, f in [0.5, 1),
 *   N2 = min(floor(M 2^N1), 2^31 - 1),
 *   y  = clip(floor((N2 q + 2^(N1-1)) / 2^N1) + zp_out, 0, 2^b - 1)
 * (round half up, as for the LayerNorm output). */
int oracle_requant_dyadic_int8(const int32_t* q, int64_t n, float s_in, float s_out,
                               int32_t zp_out, int32_t bits, int8_t* y) {
    if (n < 0 || bits < 2 || bits > 8 || !(s_in > 0.0f) || !(s_out > 0.0f)) return ORACLE_ERR_ARG;
    if (n == 0) return ORACLE_OK;
    if (!q || !y) return ORACLE_ERR_ARG;
    const int64_t half = (int64_t)1 << (bits - 1);
    const int64_t levels = ((int64_t)1 << bits) - 1;
    const int64_t zp = (int64_t)zp_out + half;      /* container -> paper grid */
    if (zp < 0 || zp > levels) return ORACLE_ERR_ARG;

    const double M = (double)s_in / (double)s_out;
    int e = 0;
    (void)frexp(M, &e);
    int64_t N1 = 31 - (int64_t)e;
    N1 = clip_i64(N1, 0, 62);
    double n2 = floor(ldexp(M, (int)N1));
    if (n2 > 2147483647.0) n2 = 2147483647.0;
    const int64_t N2 = (int64_t)n2;
    for (int64_t i = 0; i < n; ++i) {
        const __int128 prod = (__int128)N2 * (__int128)q[i];
        const __int128 w = N1 > 0 ? (prod + ((__int128)1 << (N1 - 1))) >> N1 : prod;
        const __int128 yu = w + zp;
        const int64_t yc = yu < 0 ? 0 : (yu > levels ? levels : (int64_t)yu);
        y[i] = (int8_t)(yc - half);
    }
    return ORACLE_OK;
}

/* ------------------------------------------------------------------------ */
/* Supplement A.1: quantized inference of LayerNorm with PTF                  */
/* ------------------------------------------------------------------------ */

int oracle_ptf_layernorm_int8(const int8_t* x_q, int64_t T, int32_t C, int32_t zp_in,
                              const uint8_t* alpha, int32_t K, const float* gamma,
                              const float* beta, float s_out, int32_t zp_out, int32_t bits,
                              int8_t* y_q) {
    if (T < 0 || C < 1 || bits < 2 || bits > 8 || K < 0 || K > 7 || !(s_out > 0.0f))
        return ORACLE_ERR_ARG;
    if (T == 0) return ORACLE_OK;
    if (!x_q || !alpha || !gamma || !beta || !y_q) return ORACLE_ERR_ARG;

    /* READING (containers): activations are unsigned b-bit integers in the paper
     * (eq. 2, 8).  The int8 container holds (paper value - 2^(b-1)); zero points
     * are shifted the same way.  Convert to the paper's grid first. */
    const int64_t half = (int64_t)1 << (bits - 1);
    const int64_t levels = ((int64_t)1 << bits) - 1;
    const int64_t zp = (int64_t)zp_in + half;
    const int64_t zp_o = (int64_t)zp_out + half;
    if (zp < 0 || zp > levels || zp_o < 0 || zp_o > levels) return ORACLE_ERR_ARG;

    int64_t* Xh = (int64_t*)malloc(sizeof(int64_t) * (size_t)C);
    if (!Xh) return ORACLE_ERR_ARG;

    for (int64_t t = 0; t < T; ++t) {
        const int8_t* row = x_q + t * C;

        /* Phase 1: X^_Q = (X_Q - zp) << alpha.
         * READING: alpha > K is not defined by the paper; it is clamped to K. */
        for (int32_t i = 0; i < C; ++i) {
            const int64_t XQ = (int64_t)row[i] + half;
            const int32_t a = alpha[i] < K ? alpha[i] : K;
            Xh[i] = (XQ - zp) * ((int64_t)1 << a);
        }

        /* Phase 2: M1 = sum X^_Q, M2 = sum X^_Q^2 (integers). */
        int64_t M1 = 0, M2 = 0;
        for (int32_t i = 0; i < C; ++i) {
            M1 += Xh[i];
            M2 += Xh[i] * Xh[i];
        }
        /* sigma^2 ~ (s^2/C^2)(C M2 - M1^2) and sqrt(sigma^2 + eps) ~ (s/C) sqrt(C M2 - M1^2):
         * the epsilon is dropped by the approximation. */
        const int64_t Vr = (int64_t)C * M2 - M1 * M1;

        for (int32_t i = 0; i < C; ++i) {
            /* A = s_in gamma / (s_out sqrt(sigma^2+eps)),
             * B = (beta sqrt(sigma^2+eps) - gamma mu) / (s_out sqrt(sigma^2+eps)),
             * with mu = (s/C) M1 and sqrt(sigma^2+eps) = (s/C) sqrt(Vr).  The input
             * scale s_in = s cancels:  A = gamma * C / (s_out sqrt(Vr)),
             * B = beta/s_out - gamma * M1 / (s_out sqrt(Vr)).
             * READING (floating-point order): the paper leaves A and B real.  They
             * are evaluated in IEEE double as gs = gamma/s_out, bs = beta/s_out,
             * D = sqrt(Vr), r = C/D, m = M1/D, A = gs*r, B = bs - gs*m, each
             * operation rounded on its own.
             * READING (constant row): for Vr = 0 the normalised value (X - mu)/sigma
             * is zero, so A = 0 and B = beta/s_out. */
            const double gs = (double)gamma[i] / (double)s_out;
            const double bs = (double)beta[i] / (double)s_out;
            double A, B;
            if (Vr == 0) {
                A = 0.0;
                B = bs;
            } else {
                const double D = sqrt((double)Vr);
                const double r = (double)C / D;
                const double m = (double)M1 / D;
                A = gs * r;
                B = bs - gs * m;
            }

            /* N1 = b - 1 - floor(log2|A|), N2 = floor(|A| 2^N1), A ~ sign(A) N2 / 2^N1.
             * READING: for A = 0 (gamma = 0 or a constant row) N1 = N2 = 0; N1 is
             * clamped to [0, 30] and N2 to 2^31 - 1 (never reached on sane scales). */
            int64_t N1 = 0, N2 = 0, sgn = 1;
            if (A != 0.0) {
                N1 = (int64_t)bits - 1 - (int64_t)ilogb(fabs(A));
                N1 = clip_i64(N1, 0, 30);
                const double scaled = ldexp(fabs(A), (int)N1);
                N2 = scaled >= 2147483647.0 ? 2147483647 : (int64_t)floor(scaled);
                sgn = A < 0.0 ? -1 : 1;
            }

            /* round(B 2^N1) with ties to even (READING).  READING: clamped to
             * +-2^62 so that it fits int64; any value that large saturates Y_Q. */
            const double Bs = clip_d(round_nearest(ldexp(B, (int)N1)), -0x1p62, 0x1p62);
            const int64_t Bq = (int64_t)Bs;

            /* Y_Q = round((sign(A) N2 X^_Q + round(B 2^N1)) / 2^N1) + zp_out.
             * READING: the outer rounding of this dyadic division rounds halves
             * up, floor((y + 2^(N1-1)) / 2^N1).  READING: the output is clipped
             * to the b-bit grid [0, 2^b - 1], as every activation is. */
            const int64_t y = sgn * N2 * Xh[i] + Bq;
            const int64_t w = (N1 == 0) ? y : floor_div(y + ((int64_t)1 << (N1 - 1)),
                                                         (int64_t)1 << N1);
            const int64_t YQ = clip_i64(w + zp_o, 0, levels);
            y_q[t * C + i] = (int8_t)(YQ - half);
        }
    }
    free(Xh);
    return ORACLE_OK;
}

/* ------------------------------------------------------------------------ */
/* Supplement A.2, Algorithm 1: integer-only exponential                     */
/* ------------------------------------------------------------------------ */

/* Coefficients of L(p) = a (p + b)^2 + c, the second-order fit of exp on (-ln2, 0]. */
static const double IEXP_A = 0.3585;
static const double IEXP_B = 1.353;
static const double IEXP_C = 0.344;
static const double LN2 = 0.69314718055994530942;

int oracle_iexp_constants(double s, int32_t n, oracle_iexp_consts* k) {
    if (!k || !(s > 0.0) || n < 0 || n > 62) return ORACLE_ERR_ARG;
    k->q_ln2 = (int64_t)floor(-LN2 / s);                  /* q_ln2 = floor(-ln2/s)      */
    k->q_b = (int64_t)floor(IEXP_B / s);                  /* q_b   = floor(b/s)         */
    k->q_c = (int64_t)floor(IEXP_C / ((IEXP_A * s) * s)); /* q_c   = floor(c/(a s^2))   */
    /* READING: the algorithm prints s_L <- floor(a s^2), which is 0 for any
     * useful scale; the output scale is the real a s^2. */
    k->s_L = (IEXP_A * s) * s;
    k->n = n;
    return ORACLE_OK;
}

/* I-Exp (Supplement A.2, Alg. 1).  For an input t <= 0 of scale s, clamped
 * below at n q_ln2 (READING: the depth n is not defined by the paper; it is
 * an argument, and 2^-n is then the smallest output relative to exp(0)),
 * write u = -t = z d + r with d = -q_ln2 > 0, z = floor(u / d) and
 * r in [0, d): then exp(s t) = 2^-z exp(-s r), and exp on (-ln2, 0] is
 * replaced by the quadratic L(p) = a (p + b)^2 + c, which on the integer
 * grid is s_L ((q_b - r)^2 + q_c).  The result is that polynomial value
 * scaled by 2^(n - z), with scale s_L / 2^n.
 * READING: the algorithm prints the polynomial as (q + q_b)^2 + q_c; it is
 * evaluated at the remainder, -r, as the definition of L(p) requires. */
int64_t oracle_iexp(int64_t q, const oracle_iexp_consts* k, int64_t* z_out, int64_t* qp_out) {
    const int64_t d = -k->q_ln2;
    const int64_t u_max = (int64_t)k->n * d;
    const int64_t u = -q < u_max ? -q : u_max;          /* the clamp at n q_ln2 */
    const int64_t z = u / d;                            /* u >= 0, d > 0: floor */
    const int64_t r = u - z * d;                        /* in [0, d) */
    const int64_t w = k->q_b - r;
    const int64_t poly = w * w + k->q_c;
    if (z_out) *z_out = z;
    if (qp_out) *qp_out = -r;
    return poly << (k->n - z);
}

/* ------------------------------------------------------------------------ */
/* Supplement A.2, Algorithm 2: I-Log2 and Log-Int-Softmax                   */
/* ------------------------------------------------------------------------ */

/* I-Log2 (Supplement A.2, Alg. 2): log2 r rounded to an integer at the
 * midpoint 1.5 2^M of [2^M, 2^(M+1)), M the index of the leading one of r.
 * READING: r = 1 (M = 0) has no bit below its leading one and maps to 0. */
int32_t oracle_ilog2(uint64_t r) {
    if (r == 0) return 0;
    int32_t M = 63;
    while (((r >> M) & 1u) == 0) --M;
    const int32_t round_up = (unsigned __int128)2 * r >= ((unsigned __int128)3 << M);
    return M + round_up;
}

static int lis_check(int64_t G, int32_t Lq, int32_t Lk, int32_t bits, int32_t exp_n,
                     float s_logit) {
    if (G < 0 || Lq < 0 || Lk < 1 || bits < 1 || bits > 8 || exp_n < 1 || exp_n > 30 ||
        !(s_logit > 0.0f))
        return ORACLE_ERR_ARG;
    return ORACLE_OK;
}

/* Bytes per row of stored codes: two per byte up to 4 bits, else one per byte. */
static int32_t codes_row_bytes(int32_t Lk, int32_t bits) {
    return bits <= 4 ? (Lk + 1) / 2 : Lk;
}

/* Log-Int-Softmax of one row (Supplement A.2, Alg. 2, with the clip of the
 * LIS equation in the same section): e_j = I-Exp(v_j - max_i v_i), S = sum e_j
 * (a wide integer, so it cannot wrap), and
 *     Attn_Q_j = min(I-Log2(round(S / e_j)), 2^b - 1),
 * where round(S / e_j) = floor((2 S + e_j) / (2 e_j)) (READING: ties round up;
 * the ratio is at least 1).  Attn_Q_j approximates -log2 of the softmax
 * probability e_j / S; the paper's LIS output is N - Attn_Q_j with
 * N = 2^b - 1 and scale 2^-N.  READING: Algorithm 2 omits the clip that the
 * LIS equation has; it is applied. */
static void lis_row(const int64_t* v, int32_t Lk, const oracle_iexp_consts* k, int32_t bits,
                    int64_t* e, int32_t* code) {
    int64_t vmax = v[0];
    for (int32_t j = 1; j < Lk; ++j) vmax = v[j] > vmax ? v[j] : vmax;
    unsigned __int128 S = 0;
    for (int32_t j = 0; j < Lk; ++j) {
        e[j] = oracle_iexp(v[j] - vmax, k, NULL, NULL);
        S += (unsigned __int128)e[j];
    }
    const int32_t top = (1 << bits) - 1;
    for (int32_t j = 0; j < Lk; ++j) {
        const unsigned __int128 ej = (unsigned __int128)e[j];
        const unsigned __int128 ratio = (2 * S + ej) / (2 * ej);
        const uint64_t r = ratio > (unsigned __int128)UINT64_MAX ? UINT64_MAX : (uint64_t)ratio;
        const int32_t lg = oracle_ilog2(r);
        code[j] = lg < top ? lg : top;
    }
}

int oracle_lis_softmax_log4(const int32_t* logits, int64_t G, int32_t Lq, int32_t Lk,
                            const int32_t* bias, int32_t Hb, float s_logit, int32_t bits,
                            int32_t exp_n, uint8_t* codes, int32_t ld_codes) {
    if (lis_check(G, Lq, Lk, bits, exp_n, s_logit) != ORACLE_OK) return ORACLE_ERR_ARG;
    if (ld_codes < codes_row_bytes(Lk, bits)) return ORACLE_ERR_ARG;
    if (bias && Hb < 1) return ORACLE_ERR_ARG;
    if (G == 0 || Lq == 0) return ORACLE_OK;
    if (!logits || !codes) return ORACLE_ERR_ARG;

    oracle_iexp_consts k;
    if (oracle_iexp_constants((double)s_logit, exp_n, &k) != ORACLE_OK) return ORACLE_ERR_ARG;

    int64_t* v = (int64_t*)malloc(sizeof(int64_t) * (size_t)Lk);
    int64_t* e = (int64_t*)malloc(sizeof(int64_t) * (size_t)Lk);
    int32_t* code = (int32_t*)malloc(sizeof(int32_t) * (size_t)Lk);
    if (!v || !e || !code) {
        free(v); free(e); free(code);
        return ORACLE_ERR_ARG;
    }
    for (int64_t g = 0; g < G; ++g) {
        for (int32_t i = 0; i < Lq; ++i) {
            const int32_t* q = logits + (g * Lq + i) * (int64_t)Lk;
            /* READING: a relative-position bias (Swin) is part of the logit and is
             * added before the row maximum. */
            const int32_t* bq = bias ? bias + ((g % Hb) * Lq + i) * (int64_t)Lk : NULL;
            for (int32_t j = 0; j < Lk; ++j) v[j] = (int64_t)q[j] + (bq ? bq[j] : 0);
            lis_row(v, Lk, &k, bits, e, code);
            /* READING (storage): codes of up to 4 bits two per byte, even key in
             * the low nibble; wider codes (Sec. 3.3 allows any b) one per byte. */
            uint8_t* out = codes + (g * Lq + i) * (int64_t)ld_codes;
            if (bits <= 4) {
                for (int32_t j = 0; j < Lk; j += 2) {
                    const int32_t lo = code[j];
                    const int32_t hi = (j + 1 < Lk) ? code[j + 1] : 0;
                    out[j / 2] = (uint8_t)(lo | (hi << 4));
                }
            } else {
                for (int32_t j = 0; j < Lk; ++j) out[j] = (uint8_t)code[j];
            }
        }
    }
    free(v); free(e); free(code);
    return ORACLE_OK;
}

int oracle_lis_row_exp(const int32_t* row, const int32_t* bias_row, int32_t Lk, float s_logit,
                       int32_t exp_n, int64_t* e_out, double* sum_out) {
    if (!row || !e_out || Lk < 1 || exp_n < 1 || exp_n > 30 || !(s_logit > 0.0f))
        return ORACLE_ERR_ARG;
    oracle_iexp_consts k;
    if (oracle_iexp_constants((double)s_logit, exp_n, &k) != ORACLE_OK) return ORACLE_ERR_ARG;
    int64_t mx = (int64_t)row[0] + (bias_row ? bias_row[0] : 0);
    for (int32_t j = 1; j < Lk; ++j) {
        const int64_t vj = (int64_t)row[j] + (bias_row ? bias_row[j] : 0);
        if (vj > mx) mx = vj;
    }
    double sum = 0.0;
    for (int32_t j = 0; j < Lk; ++j) {
        const int64_t vj = (int64_t)row[j] + (bias_row ? bias_row[j] : 0);
        e_out[j] = oracle_iexp(vj - mx, &k, NULL, NULL);
        sum += (double)e_out[j];
    }
    if (sum_out) *sum_out = sum;
    return ORACLE_OK;
}

/* ------------------------------------------------------------------------ */
/* Sec. 3.3 eq. (16)-(17), Supplement A.2: BitShift Attn x V                 */
/* ------------------------------------------------------------------------ */

int oracle_lis_attn_v_shift(const uint8_t* codes, int32_t ld_codes, const int8_t* v,
                            int32_t zp_v, int64_t G, int32_t Lq, int32_t Lk, int32_t d,
                            int32_t bits, int32_t* out) {
    if (G < 0 || Lq < 0 || Lk < 1 || d < 1 || bits < 1 || bits > 4 || ld_codes < (Lk + 1) / 2 ||
        zp_v < -128 || zp_v > 127)
        return ORACLE_ERR_ARG;
    if (G == 0 || Lq == 0) return ORACLE_OK;
    if (!codes || !v || !out) return ORACLE_ERR_ARG;
    /* N = 2^b - 1; Attn x V = (s_V / 2^N) * sum_j (V_Q - zp_V) << (N - Attn_Q).
     * The main-text form omits zp_V; the supplement's form includes it. */
    const int32_t N = (1 << bits) - 1;
    int rc = ORACLE_OK;
    for (int64_t g = 0; g < G; ++g) {
        for (int32_t i = 0; i < Lq; ++i) {
            const uint8_t* crow = codes + (g * Lq + i) * (int64_t)ld_codes;
            for (int32_t c = 0; c < d; ++c) {
                int64_t acc = 0;
                for (int32_t j = 0; j < Lk; ++j) {
                    const int32_t byte = crow[j / 2];
                    const int32_t attn_q = (j % 2 == 0) ? (byte & 15) : (byte >> 4);
                    const int32_t shift = N - attn_q;
                    const int64_t vq = (int64_t)v[(g * Lk + j) * (int64_t)d + c] - zp_v;
                    acc += vq * ((int64_t)1 << (shift < 0 ? 0 : shift));
                    if (shift < 0) rc = ORACLE_ERR_ARG;   /* a code above 2^b - 1 */
                }
                if (acc > INT32_MAX || acc < INT32_MIN) rc = ORACLE_ERR_RANGE;
                out[(g * Lq + i) * (int64_t)d + c] = (int32_t)(uint32_t)(uint64_t)acc;
            }
        }
    }
    return rc;
}

/* BitShift Attn x V for codes of any width b in [1, 8] (READING: the paper
 * does not say how codes wider than 4 bits multiply V; with N = 2^b - 1 the
 * integer form (V - zp) << (N - code) would need shifts of up to 255).  The
 * product is kept at the fixed output scale s_V / 2^W, W = min(2^b - 1, 44):
 *     out[g,i,c] = sum_j floor((v[g,j,c] - zp_v) 2^(W - code[g,i,j])),
 * exact (no floor acts) for every code <= W.  W = 44 covers every code
 * Log-Int-Softmax can produce for Lk <= 4096 and n <= 30: the row sum is at
 * most Lk (q_b^2 + q_c) 2^n, every I-Exp value is at least
 * min(q_b^2 + q_c, 2 ((q_b + q_ln2 + 1)^2 + q_c)) > (q_b^2 + q_c) / 2, so
 * round(S / e) < 2^43 + 1 and I-Log2 of it is at most 44.  Those products are
 * below 255 (1.5) 2^44 < 2^53 in magnitude (sum_j 2^-code_j < 1.5 without a
 * clip).  A code above W (only from codes not made by Log-Int-Softmax)
 * contributes the floor of its right shift; a sum that leaves int64 (again
 * only for such codes) wraps modulo 2^64.  For b <= 4 this is
 * oracle_lis_attn_v_shift widened to int64.  Codes are stored as
 * oracle_lis_softmax_log4 writes them (nibbles for b <= 4, bytes above). */
int oracle_lis_attn_v_shift_wide(const uint8_t* codes, int32_t ld_codes, const int8_t* v,
                                 int32_t zp_v, int64_t G, int32_t Lq, int32_t Lk, int32_t d,
                                 int32_t bits, int64_t* out) {
    if (G < 0 || Lq < 0 || Lk < 1 || d < 1 || bits < 1 || bits > 8 ||
        ld_codes < codes_row_bytes(Lk, bits) || zp_v < -128 || zp_v > 127)
        return ORACLE_ERR_ARG;
    if (G == 0 || Lq == 0) return ORACLE_OK;
    if (!codes || !v || !out) return ORACLE_ERR_ARG;
    const int32_t N = (1 << bits) - 1;
    const int32_t W = N < 44 ? N : 44;
    for (int64_t g = 0; g < G; ++g) {
        for (int32_t i = 0; i < Lq; ++i) {
            const uint8_t* crow = codes + (g * Lq + i) * (int64_t)ld_codes;
            for (int32_t c = 0; c < d; ++c) {
                uint64_t acc = 0;      /* two's complement sum, modulo 2^64 */
                for (int32_t j = 0; j < Lk; ++j) {
                    int32_t attn_q;
                    if (bits <= 4) attn_q = (j % 2 == 0) ? (crow[j / 2] & 15) : (crow[j / 2] >> 4);
                    else attn_q = crow[j];
                    const int64_t vq = (int64_t)v[(g * Lk + j) * (int64_t)d + c] - zp_v;
                    int64_t term;
                    if (attn_q <= W) term = vq * ((int64_t)1 << (W - attn_q));
                    else term = floor_div(vq, (int64_t)1 << (attn_q - W < 62 ? attn_q - W : 62));
                    acc += (uint64_t)term;
                }
                out[(g * Lq + i) * (int64_t)d + c] = (int64_t)acc;
            }
        }
    }
    return ORACLE_OK;
}

int oracle_lis_attention_head(const int32_t* logits, const int32_t* bias, int32_t Hb,
                              int64_t G, int32_t Lq, int32_t Lk, float s_logit, int32_t bits,
                              int32_t exp_n, const int8_t* v, int32_t zp_v, int32_t d,
                              int32_t* out, uint8_t* codes_out, int32_t ld_codes) {
    if (lis_check(G, Lq, Lk, bits, exp_n, s_logit) != ORACLE_OK || d < 1 || bits > 4)
        return ORACLE_ERR_ARG;
    const int32_t ld = (Lk + 1) / 2;
    if (codes_out && ld_codes < ld) return ORACLE_ERR_ARG;
    if (G == 0 || Lq == 0) return ORACLE_OK;
    uint8_t* tmp = (uint8_t*)malloc((size_t)(G * Lq) * (size_t)ld);
    if (!tmp) return ORACLE_ERR_ARG;
    int rc = oracle_lis_softmax_log4(logits, G, Lq, Lk, bias, Hb, s_logit, bits, exp_n, tmp, ld);
    if (rc == ORACLE_OK)
        rc = oracle_lis_attn_v_shift(tmp, ld, v, zp_v, G, Lq, Lk, d, bits, out);
    if (rc == ORACLE_OK && codes_out)
        for (int64_t r = 0; r < G * Lq; ++r)
            memcpy(codes_out + r * ld_codes, tmp + r * ld, (size_t)ld);
    free(tmp);
    return rc;
}

/* ------------------------------------------------------------------------ */
/* Integer-only MSA (Sec. 3.3, its Fig. 4): int8 Q K^T, then LIS and BitShift */
/* ------------------------------------------------------------------------ */

/* The attention logits of the integer-only dataflow: the MinMax-quantized
 * MatMul of Sec. 3.1 (its int GEMMs for MatMul) between the query and key
 * activations, exact in integers:
 *   logit[g,i,j] = sum_c (q[g,i,c] - zp_q) (k[g,j,c] - zp_k)
 * with q, k and the zero points in the int8 container (the offset 2^(b-1)
 * cancels in each difference).  Its scale, s_q s_k (with any 1/sqrt(dk) of
 * the softmax folded in), is the s_logit of Log-Int-Softmax, which follows
 * together with the BitShift product as in oracle_lis_attention_head. */
int oracle_qk_logits(const int8_t* q, const int8_t* k, int32_t zp_q, int32_t zp_k, int64_t G,
                     int32_t Lq, int32_t Lk, int32_t dk, int32_t* logits) {
    if (G < 0 || Lq < 0 || Lk < 1 || dk < 1) return ORACLE_ERR_ARG;
    if (zp_q < -128 || zp_q > 127 || zp_k < -128 || zp_k > 127) return ORACLE_ERR_ARG;
    for (int64_t g = 0; g < G; ++g)
        for (int32_t i = 0; i < Lq; ++i)
            for (int32_t j = 0; j < Lk; ++j) {
                int64_t acc = 0;
                const int8_t* qi = q + (g * Lq + i) * (int64_t)dk;
                const int8_t* kj = k + (g * Lk + j) * (int64_t)dk;
                for (int32_t c = 0; c < dk; ++c)
                    acc += ((int64_t)qi[c] - zp_q) * ((int64_t)kj[c] - zp_k);
                if (acc > INT32_MAX || acc < INT32_MIN) return ORACLE_ERR_RANGE;
                logits[(g * Lq + i) * (int64_t)Lk + j] = (int32_t)acc;
            }
    return ORACLE_OK;
}

int oracle_lis_attention_qk(const int8_t* q, const int8_t* k, int32_t zp_q, int32_t zp_k,
                            int32_t dk, const int32_t* bias, int32_t Hb, int64_t G, int32_t Lq,
                            int32_t Lk, float s_logit, int32_t bits, int32_t exp_n,
                            const int8_t* v, int32_t zp_v, int32_t d, int32_t* out) {
    if (G < 0 || Lq < 0 || Lk < 1 || dk < 1) return ORACLE_ERR_ARG;
    if (G == 0 || Lq == 0) return ORACLE_OK;
    int32_t* logits = (int32_t*)malloc(sizeof(int32_t) * (size_t)(G * Lq) * (size_t)Lk);
    if (!logits) return ORACLE_ERR_ARG;
    int rc = oracle_qk_logits(q, k, zp_q, zp_k, G, Lq, Lk, dk, logits);
    if (rc == ORACLE_OK)
        rc = oracle_lis_attention_head(logits, bias, Hb, G, Lq, Lk, s_logit, bits, exp_n, v, zp_v,
                                       d, out, NULL, 0);
    free(logits);
    return rc;
}
