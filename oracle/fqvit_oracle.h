/*
 * fqvit_oracle.h -- CPU oracle for the integer hot path of FQ-ViT
 * (Lin et al., "FQ-ViT: Post-Training Quantization for Fully Quantized
 * Vision Transformer", IJCAI 2022).
 *
 * TEST INFRASTRUCTURE ONLY.  This library exists to check the HIP library
 * against the paper.  Only the test suite, the smoke check and the CPU
 * baseline leg of the benchmark may load it; the product path never does,
 * and the two share no code, header, table or constant generator.
 *
 * All pointers are HOST pointers.  Every integer tensor uses the same
 * containers as the HIP library's C ABI (see the comments below), but the
 * arithmetic is written out on the paper's own unsigned grids, step by
 * step, in plain scalar C with exact integers, plus IEEE double for the
 * real-valued quantities the paper leaves as reals.  Where the paper is
 * silent or its printed formula is garbled, the choice made is marked
 * "READING" in fqvit_oracle.c.
 *
 * Parity status: every function is pinned by the CPU tests except where a
 * function's comment says "parity unpinned".
 */
#ifndef FQVIT_ORACLE_H
#define FQVIT_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Return codes (0 = success). */
enum {
    ORACLE_OK = 0,
    ORACLE_ERR_ARG = 1,      /* invalid argument                          */
    ORACLE_ERR_RANGE = 2     /* a result does not fit its output type      */
};

/* ---- Sec. 3.1, eq. (3)-(5): uniform MinMax quantizer ------------------ */

/* s = (u - l)/(2^b - 1), zp = clip(round(-l/s), 0, 2^b - 1) over x[0..n). */
int oracle_minmax_params(const double* x, int64_t n, int32_t b, double* s, int32_t* zp);
/* q = clip(round(x/s) + zp, 0, 2^b - 1) on the unsigned grid. */
int oracle_minmax_quantize(const double* x, int64_t n, double s, int32_t zp, int32_t b,
                           int32_t* q);

/* ---- Sec. 3.2, eq. (8)-(11): Power-of-Two-Factor quantizer ------------ */

/* Layer-wise s (eq. 9) and zp (eq. 10) over a row-major [T, C] tensor. */
int oracle_ptf_params(const double* x, int64_t T, int32_t C, int32_t b, int32_t K,
                      double* s, int32_t* zp);
/* Per-channel alpha by the argmin of eq. (11) over {0..K}: each channel's
 * error is the exact sum of the exact squared errors, so no summation order
 * enters; ties go to the smallest alpha.  T <= 2^26. */
int oracle_ptf_alpha(const double* x, int64_t T, int32_t C, double s, int32_t zp,
                     int32_t b, int32_t K, uint8_t* alpha);
/* The exact errors themselves, err[c (K+1) + a]: the exact value rounded to
 * a double (within one unit in the last place) and, if err_lo is non-null,
 * err_lo[c (K+1) + a] the rest of the exact value, rounded. */
int oracle_ptf_alpha_errors(const double* x, int64_t T, int32_t C, double s, int32_t zp,
                            int32_t b, int32_t K, double* err, double* err_lo);
/* X_Q = clip(round(X / (2^alpha_c s)) + zp, 0, 2^b - 1) (eq. 8), unsigned grid. */
int oracle_ptf_quantize(const double* x, int64_t T, int32_t C, double s, int32_t zp,
                        const uint8_t* alpha, int32_t b, int32_t* q);

/* ---- Dyadic requantization (the integer form of Supplement A.1) ------ */

/* y = clip(round((N2 / 2^N1) q) + zp_out) with N2 / 2^N1 the 31-bit dyadic
 * form of s_in / s_out; y and zp_out in the int8 container of b-bit values
 * (value - 2^(b-1)).  bits in [2, 8]. */
int oracle_requant_dyadic_int8(const int32_t* q, int64_t n, float s_in, float s_out,
                               int32_t zp_out, int32_t bits, int8_t* y);

/* ---- Supplement A.1: integer-only PTF LayerNorm ---------------------- */

/* x_q, y_q: row-major [T, C] int8 containers holding (paper value - 2^(bits-1));
 * zp_in, zp_out are shifted the same way.  alpha[C] is clamped to K.
 * gamma, beta: [C] float.  s_out > 0.  bits in [2, 8], K in [0, 7]. */
int oracle_ptf_layernorm_int8(const int8_t* x_q, int64_t T, int32_t C, int32_t zp_in,
                              const uint8_t* alpha, int32_t K, const float* gamma,
                              const float* beta, float s_out, int32_t zp_out, int32_t bits,
                              int8_t* y_q);

/* ---- Supplement A.2, Algorithm 1: I-Exp ------------------------------ */

typedef struct {
    int64_t q_ln2;   /* floor(-ln2 / s)          */
    int64_t q_b;     /* floor(b / s),  b = 1.353  */
    int64_t q_c;     /* floor(c / (a s^2)), a = 0.3585, c = 0.344 */
    double s_L;      /* a s^2                     */
    int32_t n;       /* clamp depth               */
} oracle_iexp_consts;

int oracle_iexp_constants(double s, int32_t n, oracle_iexp_consts* k);
/* i-exp of one non-positive quantized input q; output scale s_L / 2^n.
 * If z_out is non-null it receives z, if qp_out is non-null it receives q_p. */
int64_t oracle_iexp(int64_t q, const oracle_iexp_consts* k, int64_t* z_out, int64_t* qp_out);

/* ---- Supplement A.2, Algorithm 2: I-Log2 and Log-Int-Softmax --------- */

/* M + chi with M the index of the most significant 1 bit of q, chi the bit below it. */
int32_t oracle_ilog2(uint64_t q);

/* logits: [G, Lq, Lk] int32; bias: nullable [Hb, Lq, Lk] int32, unit g uses head g % Hb.
 * codes: Attn_Q in [0, 2^bits - 1]; for bits <= 4 two per byte (even key in the
 * low nibble), row stride ld_codes >= ceil(Lk / 2) bytes; for bits in [5, 8] one
 * per byte, ld_codes >= Lk.  Bytes past the row's codes are not written.
 * bits in [1, 8]. */
int oracle_lis_softmax_log4(const int32_t* logits, int64_t G, int32_t Lq, int32_t Lk,
                            const int32_t* bias, int32_t Hb, float s_logit, int32_t bits,
                            int32_t exp_n, uint8_t* codes, int32_t ld_codes);

/* The I-Exp values e_j of one row (after adding bias and subtracting the row max)
 * and their sum, for the secondary checks against a float softmax. */
int oracle_lis_row_exp(const int32_t* row, const int32_t* bias_row, int32_t Lk, float s_logit,
                       int32_t exp_n, int64_t* e_out, double* sum_out);

/* ---- Sec. 3.3 and Supplement A.2: BitShift Attn x V ------------------ */

/* out[g,i,c] = sum_j (v[g,j,c] - zp_v) << ((2^bits - 1) - code[g,i,j]).
 * v: [G, Lk, d] int8 container; out: [G, Lq, d] int32.  bits in [1, 4].
 * Returns ORACLE_ERR_RANGE if a sum does not fit int32. */
int oracle_lis_attn_v_shift(const uint8_t* codes, int32_t ld_codes, const int8_t* v,
                            int32_t zp_v, int64_t G, int32_t Lq, int32_t Lk, int32_t d,
                            int32_t bits, int32_t* out);

/* The same product for codes of any width b in [1, 8], as int64 at the output
 * scale s_V / 2^W, W = min(2^b - 1, 44): out = sum_j floor((v - zp_v)
 * 2^(W - code)), exact for codes <= W (every code Log-Int-Softmax produces);
 * modulo 2^64 if a sum leaves int64 (never for those codes).
 * codes: nibbles for b <= 4, one byte per code above. */
int oracle_lis_attn_v_shift_wide(const uint8_t* codes, int32_t ld_codes, const int8_t* v,
                                 int32_t zp_v, int64_t G, int32_t Lq, int32_t Lk, int32_t d,
                                 int32_t bits, int64_t* out);

/* Log-Int-Softmax followed by BitShift Attn x V. codes_out is nullable. */
int oracle_lis_attention_head(const int32_t* logits, const int32_t* bias, int32_t Hb,
                              int64_t G, int32_t Lq, int32_t Lk, float s_logit, int32_t bits,
                              int32_t exp_n, const int8_t* v, int32_t zp_v, int32_t d,
                              int32_t* out, uint8_t* codes_out, int32_t ld_codes);

/* ---- Sec. 3.3, Fig. 4: integer-only MSA from int8 Q and K ------------- */

/* logits[g,i,j] = sum_c (q[g,i,c] - zp_q)(k[g,j,c] - zp_k); q: [G, Lq, dk],
 * k: [G, Lk, dk] int8 containers, zero points in container form. */
int oracle_qk_logits(const int8_t* q, const int8_t* k, int32_t zp_q, int32_t zp_k, int64_t G,
                     int32_t Lq, int32_t Lk, int32_t dk, int32_t* logits);
/* oracle_qk_logits, then oracle_lis_attention_head on those logits. */
int oracle_lis_attention_qk(const int8_t* q, const int8_t* k, int32_t zp_q, int32_t zp_k,
                            int32_t dk, const int32_t* bias, int32_t Hb, int64_t G, int32_t Lq,
                            int32_t Lk, float s_logit, int32_t bits, int32_t exp_n,
                            const int8_t* v, int32_t zp_v, int32_t d, int32_t* out);

#ifdef __cplusplus
}
#endif
#endif
