/*
 * fqvit.h -- C ABI of the MI355X (gfx950) library for the integer hot path of
 * FQ-ViT (Lin et al., "FQ-ViT: Post-Training Quantization for Fully Quantized
 * Vision Transformer", IJCAI 2022): Power-of-Two-Factor LayerNorm and
 * Log-Int-Softmax attention.
 *
 * Conventions shared by every entry point
 *   - Tensor arguments are DEVICE pointers into memory the caller owns (for
 *     example allocated through torch).  The library allocates nothing, never
 *     synchronises, and enqueues its kernels on `stream` (a hipStream_t; NULL
 *     is the default stream).  It keeps no state between calls apart from the
 *     per-thread timing events of fq_time_next_call and the fixed device array
 *     of ptf_calibrate_noalloc.  It is re-entrant (ptf_calibrate_noalloc: see
 *     its note on overlapping calls).
 *   - Scalars are passed by value.  Tensors are dense and row-major with the
 *     shapes given below; a tensor is read or written only inside the extent
 *     its shape gives.
 *   - Every argument is validated on the host before anything is enqueued.  A
 *     failing check returns its status code and enqueues nothing.  Empty
 *     tensors (T, G or Lq equal to 0) return FQ_OK and enqueue nothing.
 *   - Integer outputs are a pure function of the arguments (no atomics, no
 *     order dependence): the same call gives the same bits every time.
 *   - Quantized activations live on the paper's unsigned b-bit grid
 *     {0 .. 2^b - 1} (Sec. 3.1, eq. 2).  The int8 containers used here hold
 *     (paper value - 2^(b-1)); zero points are shifted the same way.  Every
 *     formula uses only X_Q - zp, so results are identical on either grid.
 */
#ifndef FQVIT_H
#define FQVIT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum fq_status {
    FQ_OK = 0,
    FQ_ERR_NULL = 1,      /* a required pointer is NULL                              */
    FQ_ERR_SHAPE = 2,     /* a size is out of the supported range                    */
    FQ_ERR_PARAM = 3,     /* a scalar parameter is out of range                      */
    FQ_ERR_HEADROOM = 4,  /* the exact integer sums could overflow 64 bits           */
    FQ_ERR_HIP = 5,       /* the HIP runtime rejected a launch                       */
    FQ_ERR_SCRATCH = 6    /* the call needs more than the fixed device scratch holds */
} fq_status;

/* Static, human-readable name of a status code (never NULL). */
const char* fq_status_str(int status);

/* Library version as major * 10000 + minor * 100 + patch. */
int32_t fq_version(void);

/*
 * Instrumentation, not part of the method.  Attaches two caller-created HIP
 * events (hipEvent_t, from hipEventCreate; either may be NULL) to the kernel
 * launched by the next entry-point call made on the calling thread: `start`
 * then records that kernel's start and `stop` its end (hipExtLaunchKernel
 * semantics), so hipEventElapsedTime gives the kernel's own duration with no
 * extra packets on the stream.  Every other entry point launches one kernel.
 * ptf_calibrate, which launches four kernels, records `start` on the first and
 * `stop` on the last, so the interval covers the whole calibration.
 * The events are consumed by that next call whatever it returns; a call that
 * enqueues nothing (empty tensors, failed validation) leaves them unrecorded.
 * Always returns FQ_OK.
 */
fq_status fq_time_next_call(void* start_event, void* stop_event);

/*
 * PTF LayerNorm, integer-only (Sec. 3.2, eq. 12 for the shift; Supplement A.1
 * for the statistics M1, M2, the factors A and B, their dyadic form N2 / 2^N1
 * and the output Y_Q).
 *
 *   x_q     [T, C] int8 container of the PTF-quantized input X_Q.
 *   zp_in   layer-wise zero point, container form, in [-2^(b-1), 2^(b-1) - 1].
 *   alpha   [C] uint8 power-of-two factors; values above K are clamped to K.
 *   K       0..7 (the paper uses 3).
 *   gamma, beta  [C] float affine parameters.
 *   s_out   output scale (> 0, finite); zp_out output zero point (container).
 *   bits    b in [2, 8]; the output is clipped to the b-bit grid.
 *   y_q     [T, C] int8 container output.
 * The input scale cancels from A and B and is therefore not an argument.
 * Per row: X^ = (X_Q - zp) << alpha, M1 = sum X^, M2 = sum X^^2,
 * V = C M2 - M1^2; in IEEE double, D = sqrt(V), r = C / D, m = M1 / D,
 * A = (gamma/s_out) r, B = beta/s_out - (gamma/s_out) m (each operation
 * rounded on its own; A = 0 and B = beta/s_out when V = 0);
 * N1 = clamp(b - 1 - floor(log2|A|), 0, 30), N2 = min(floor(|A| 2^N1), 2^31 - 1)
 * (both 0 when A = 0); Y = clip(floor((sign(A) N2 X^ + rint(B 2^N1)
 * + 2^(N1-1)) / 2^N1) + zp_out) (no half term when N1 = 0).
 * Errors: FQ_ERR_NULL (x_q, alpha, gamma, beta or y_q NULL with T > 0),
 * FQ_ERR_SHAPE (T < 0, C outside [1, 8192]), FQ_ERR_PARAM (bits, K, s_out or a
 * zero point out of range).
 */
fq_status ptf_layernorm_int8(const int8_t* x_q, int64_t T, int32_t C, int32_t zp_in,
                             const uint8_t* alpha, int32_t K, const float* gamma,
                             const float* beta, float s_out, int32_t zp_out, int32_t bits,
                             int8_t* y_q, void* stream);

/*
 * Log-Int-Softmax codes (Supplement A.2: Algorithm 1, I-Exp; Algorithm 2,
 * I-Log2 and Log-Int-Softmax; the clip of the LIS equation in the same
 * section).
 *
 *   logits  [G, Lq, Lk] int32 attention logits with scale s_logit
 *           (G = attention units, e.g. batch x windows x heads).
 *   bias    NULL or [Hb, Lq, Lk] int32 added to the logits of unit g from
 *           plane g % Hb before the row maximum (Swin relative-position bias:
 *           Hb = heads; with units ordered (image, window, head), a shifted-
 *           window mask is folded in by passing the sum of mask and bias as
 *           [windows, heads, Lq, Lk] with Hb = windows x heads).
 *   s_logit in [1e-4, 0.5].
 *   bits    code width b in [1, 8]; codes are Attn_Q in [0, 2^b - 1] and the
 *           LIS output of the paper is N - Attn_Q with N = 2^b - 1, scale 2^-N.
 *   exp_n   I-Exp clamp depth n in [1, 30]: inputs below n q_ln2 are clamped.
 *   codes   [G, Lq, ld_codes] uint8 output.  b <= 4: two codes per byte, the
 *           even key in the low nibble, an odd row's last high nibble 0, bytes
 *           at and beyond ceil(Lk/2) in each row not written.  b >= 5: one
 *           code per byte, bytes at and beyond Lk not written.
 * Per row: t_j = v_j - max v, e_j = I-Exp(t_j) with q_ln2 = floor(-ln2/s),
 * q_b = floor(1.353/s), q_c = floor(0.344/((0.3585 s) s)) in IEEE double,
 * S = sum e_j, Attn_Q_j = min(I-Log2(floor((2S + e_j) / (2 e_j))), 2^b - 1).
 * Errors: FQ_ERR_NULL (logits or codes NULL with G Lq > 0), FQ_ERR_SHAPE
 * (G or Lq < 0, Lk outside [1, 4096], ld_codes below ceil(Lk/2) for b <= 4 or
 * Lk for b >= 5, Hb < 1 with a bias), FQ_ERR_PARAM (bits, exp_n or s_logit
 * out of range), FQ_ERR_HEADROOM
 * ((2 Lk + 1) (q_b^2 + q_c) 2^n >= 2^63).
 * Precondition (not checked): |logit + bias| < 2^30.
 */
fq_status lis_softmax_log4(const int32_t* logits, int64_t G, int32_t Lq, int32_t Lk,
                           const int32_t* bias, int32_t Hb, float s_logit, int32_t bits,
                           int32_t exp_n, uint8_t* codes, int32_t ld_codes, void* stream);

/*
 * BitShift Attn x V (Sec. 3.3, eq. 16-17, and its zero-point form in
 * Supplement A.2):
 *   out[g, i, c] = sum_j (v[g, j, c] - zp_v) << ((2^b - 1) - code[g, i, j]).
 *
 *   codes   [G, Lq, ld_codes] packed codes as written by lis_softmax_log4.
 *   v       [G, Lk, d] int8, zero point zp_v in [-128, 127].
 *   bits    b in [1, 4] (shifts of at most 15).
 *   out     [G, Lq, d] int32, scale s_V / 2^(2^b - 1).
 * The sum is exact; it wraps modulo 2^32 only if it leaves int32, which codes
 * produced by Log-Int-Softmax never do for Lk <= 4096.  Codes above 2^b - 1
 * (never written by lis_softmax_log4) give an unspecified result.
 * Errors: FQ_ERR_NULL, FQ_ERR_SHAPE (G or Lq < 0, Lk outside [1, 4096], d
 * outside [1, 256], ld_codes < ceil(Lk/2)), FQ_ERR_PARAM (bits, zp_v).
 */
fq_status lis_attn_v_shift(const uint8_t* codes, int32_t ld_codes, const int8_t* v,
                           int32_t zp_v, int64_t G, int32_t Lq, int32_t Lk, int32_t d,
                           int32_t bits, int32_t* out, void* stream);

/*
 * BitShift Attn x V for codes of any width b in [1, 8], including the 8-bit
 * attention maps of the paper's 8/8/8 setting (Sec. 3.3; its Table 1).  The
 * paper does not say how codes wider than 4 bits multiply V: with
 * N = 2^b - 1 the integer form (V - zp) << (N - code) would need shifts of up
 * to 255.  This product keeps the fixed output scale s_V / 2^W with
 * W = min(2^b - 1, 44):
 *   out[g, i, c] = sum_j floor((v[g, j, c] - zp_v) 2^(W - code[g, i, j])),
 * which is exact (no floor acts) for every code <= W.  Log-Int-Softmax never
 * produces a code above 44 for Lk <= 4096 and n <= 30 (round(S / e) stays
 * below 2^43 + 1), so its products are exact, and below 255 (1.5) 2^44 in
 * magnitude; for b <= 4 the result is lis_attn_v_shift's widened to int64.
 * A code above W (not one made by Log-Int-Softmax) contributes the floor of
 * its shifted value, and a sum that leaves int64 (again only for such codes)
 * wraps modulo 2^64.
 *
 *   codes   [G, Lq, ld_codes] as written by lis_softmax_log4 with the same
 *           bits: nibbles for b <= 4 (ld_codes >= ceil(Lk/2)), one byte per
 *           code for b >= 5 (ld_codes >= Lk).
 *   v       [G, Lk, d] int8, zero point zp_v in [-128, 127].
 *   out     [G, Lq, d] int64, scale s_V / 2^W.
 * Errors: FQ_ERR_NULL, FQ_ERR_SHAPE (G or Lq < 0, Lk outside [1, 4096], d
 * outside [1, 256], ld_codes below the row's bytes), FQ_ERR_PARAM (bits, zp_v).
 */
fq_status lis_attn_v_shift_wide(const uint8_t* codes, int32_t ld_codes, const int8_t* v,
                                int32_t zp_v, int64_t G, int32_t Lq, int32_t Lk, int32_t d,
                                int32_t bits, int64_t* out, void* stream);

/*
 * Fused Log-Int-Softmax and BitShift Attn x V, the integer-only attention of
 * Sec. 3.3 (the MSA dataflow of its Fig. 4): the same results as
 * lis_softmax_log4 followed by lis_attn_v_shift, with the codes kept on chip.
 * Arguments as in those two calls (bits in [1, 4]); d in [1, 256]; codes_out
 * is NULL or a [G, Lq, ld_codes] buffer that also receives the codes.
 */
fq_status lis_attention_head(const int32_t* logits, const int32_t* bias, int32_t Hb,
                             int64_t G, int32_t Lq, int32_t Lk, float s_logit, int32_t bits,
                             int32_t exp_n, const int8_t* v, int32_t zp_v, int32_t d,
                             int32_t* out, uint8_t* codes_out, int32_t ld_codes, void* stream);

/*
 * Integer-only multi-head self-attention from int8 queries and keys: the
 * MinMax-quantized MatMul of Sec. 3.1 between Q and K (an integer GEMM),
 * Log-Int-Softmax and the BitShift Attn x V of Sec. 3.3 (the dataflow of its
 * Fig. 4), with the logits and codes kept on chip:
 *   logit[g,i,j] = sum_c (q[g,i,c] - zp_q)(k[g,j,c] - zp_k) (+ bias),
 * then exactly lis_attention_head on those logits.  Log-Int-Softmax depends
 * only on the differences of a row's logits, so the result does not depend on
 * zp_k (it is still validated); the kernel drops the per-query terms.
 *
 *   q       [G, Lq, dk] int8 container, 16-byte aligned; zp_q in [-128, 127].
 *   k       [G, Lk, dk] int8 container, 16-byte aligned; zp_k in [-128, 127].
 *   dk      32 or 64.
 *   bias, Hb, s_logit, bits (in [1, 4]), exp_n, v, zp_v, out: as in
 *           lis_attention_head;
 *           s_logit is the scale of the logits (s_q s_k, with any 1/sqrt(dk)
 *           of the softmax folded in).
 * Supported: Lk in [1, 640], d in [1, 64] (rows of more than 224 keys: the
 * logits are recomputed from K in each pass instead of held).
 * Errors: FQ_ERR_NULL, FQ_ERR_SHAPE (sizes, dk, or bias with Hb < 1),
 * FQ_ERR_PARAM (zero points, bits, exp_n, s_logit, or misaligned q / k),
 * FQ_ERR_HEADROOM.
 */
fq_status lis_attention_qk(const int8_t* q, const int8_t* k, int32_t zp_q, int32_t zp_k,
                           int32_t dk, const int32_t* bias, int32_t Hb, int64_t G, int32_t Lq,
                           int32_t Lk, float s_logit, int32_t bits, int32_t exp_n,
                           const int8_t* v, int32_t zp_v, int32_t d, int32_t* out, void* stream);

/*
 * PTF calibration (Sec. 3.2): the layer-wise scale and zero point of eq. (9),
 * (10) from the minimum and maximum of x, then each channel's power-of-two
 * factor alpha_c by the argmin of eq. (11) over {0 .. K}, the squared error of
 * the quantizer of eq. (8) itself (its zero point and clip included).
 *
 *   x          [T, C] float activations (finite), T in [0, 65535 * 64].
 *   bits       b in [2, 8]; K in [0, 7] (the paper uses 3).
 *   s          device double (out): s = (max - min) / (2^b - 1) / 2^K.
 *   zp         device int32 (out), container form: clip(rint(-min / (2^K s)),
 *              0, 2^b - 1) - 2^(b-1).
 *   alpha      [C] uint8 (out).
 *   workspace  device scratch of at least fq_ptf_calibrate_workspace_bytes(T,
 *              C, K) bytes, owned by the caller; its contents on entry do not
 *              matter and on return are unspecified.
 * Every operation is rounded in binary64 as written; each channel's squared
 * errors are summed in blocks of 64 consecutive rows, in order, and the block
 * sums added in order, so alpha is a pure function of x; ties of those sums go
 * to the smallest alpha.  Tie rule against the exact argmin of eq. (11): with
 * E_a the exact error of candidate a and B_a = (T + 8) 2^-53
 * sum_t (|x_tc| + 2 |deq_a(x_tc)|)^2 the bound on the rounding of its sum,
 * alpha_c is the exact argmin (ties to the smallest) unless another candidate
 * a has E_a - E_best <= B_a + B_best, in which case it may be a.  A tensor
 * whose maximum equals its minimum gets s = 0, the
 * zero point 0 of the paper's grid and alpha = 0.  T = 0 enqueues nothing and
 * leaves the outputs untouched.
 * Errors: FQ_ERR_NULL, FQ_ERR_SHAPE (T outside [0, 65535 * 64], C outside
 * [1, 8192]), FQ_ERR_PARAM (bits, K, or a workspace that is too small).
 */
size_t fq_ptf_calibrate_workspace_bytes(int64_t T, int32_t C, int32_t K);
fq_status ptf_calibrate(const float* x, int64_t T, int32_t C, int32_t bits, int32_t K, double* s,
                        int32_t* zp, uint8_t* alpha, void* workspace, size_t workspace_bytes,
                        void* stream);

/*
 * ptf_calibrate for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation): the
 * same kernels and results, with the workspace taken from a fixed device
 * array of FQ_NOALLOC_SCRATCH_BYTES that the library holds on each GPU it runs
 * on until the process ends.  This call allocates nothing (no hipMalloc, no
 * hipFree, no allocating library routine); on its first call on a device it
 * looks up that device's copy of the array (hipGetSymbolAddress).
 *   x, T, C, bits, K, s, zp, alpha: as ptf_calibrate.
 * Every call on one GPU shares that GPU's array, so calls that overlap on one
 * GPU (different streams, or host threads, without ordering between them)
 * race and give undefined results; calls ordered on one stream are safe.  The
 * array's contents on entry do not matter.
 * Errors: as ptf_calibrate, and FQ_ERR_SCRATCH when
 * fq_ptf_calibrate_workspace_bytes(T, C, K) exceeds FQ_NOALLOC_SCRATCH_BYTES
 * (nothing enqueued); FQ_ERR_HIP if the array cannot be looked up.
 */
#define FQ_NOALLOC_SCRATCH_BYTES ((size_t)8 << 20)
fq_status ptf_calibrate_noalloc(const float* x, int64_t T, int32_t C, int32_t bits, int32_t K,
                                double* s, int32_t* zp, uint8_t* alpha, void* stream);

/*
 * PTF quantizer (Sec. 3.2, eq. 8): X_Q = clip(rint(x / (2^alpha_c s)) + zp,
 * 0, 2^b - 1), in binary64, stored in the int8 container.
 *
 *   x      [T, C] float; s, zp: device scalars as written by ptf_calibrate
 *          (zp in container form); alpha [C] uint8; bits b in [2, 8].
 *   x_q    [T, C] int8 container output (the input of ptf_layernorm_int8).
 * s <= 0 (a degenerate calibration) stores zp everywhere.
 * Errors: FQ_ERR_NULL, FQ_ERR_SHAPE (T < 0, C outside [1, 8192]),
 * FQ_ERR_PARAM (bits).
 */
fq_status ptf_quantize_int8(const float* x, int64_t T, int32_t C, const double* s,
                            const int32_t* zp, const uint8_t* alpha, int32_t bits, int8_t* x_q,
                            void* stream);

/*
 * Dyadic requantization of an int32 accumulator to a b-bit activation, the
 * integer-only form of Supplement A.1 (a real multiplier replaced by
 * N2 / 2^N1 and a rounding shift), e.g. for the BitShift Attn x V output of
 * lis_attention_head (scale s_V / 2^(2^b - 1)) feeding the next layer.
 *
 *   q       [n] int32 with scale s_in.
 *   s_in, s_out  positive finite scales; zp_out the output zero point,
 *           container form.  bits b in [2, 8].
 *   y       [n] int8 container output.
 * With M = s_in / s_out in binary64, M = f 2^e (f in [0.5, 1)),
 * N1 = clamp(31 - e, 0, 62), N2 = min(floor(M 2^N1), 2^31 - 1):
 * y = clip(floor((N2 q + 2^(N1-1)) / 2^N1) + zp_out) (no half term when
 * N1 = 0), exact in 64-bit integers.
 * Errors: FQ_ERR_NULL, FQ_ERR_SHAPE (n < 0), FQ_ERR_PARAM (bits, a scale or
 * zp_out out of range).
 */
fq_status requant_dyadic_int8(const int32_t* q, int64_t n, float s_in, float s_out,
                              int32_t zp_out, int32_t bits, int8_t* y, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* FQVIT_H */
