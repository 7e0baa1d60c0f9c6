// C ABI of libfqvit (declared in include/fqvit.h): argument validation, the
// host-side integer constants of I-Exp, and the kernel launches.  Nothing here
// allocates or synchronises; the only state is the per-thread pair of timing
// events of fq_time_next_call, consumed by the next entry-point call.
#include "fqvit.h"

#include <cmath>
#include <cstdint>

#include "fqvit_internal.h"

namespace {

constexpr int32_t kMaxC = 8192;
constexpr int32_t kMaxLk = 4096;
constexpr int32_t kMaxD = 256;
// The alpha search's grid has one y index per block of 64 rows: at most
// 65535 of them.
constexpr int64_t kMaxCalibT = (int64_t)65535 * 64;

fq_status from_hip(hipError_t e) { return e == hipSuccess ? FQ_OK : FQ_ERR_HIP; }

thread_local fqvit::LaunchEvents t_events;

// Clears the timing events when an entry point returns, whatever the path.
struct ConsumeEvents {
    ~ConsumeEvents() { t_events = fqvit::LaunchEvents{}; }
};

// Integer constants of Algorithm 1 (Supplement A.2) for input scale s, plus the
// bounds that let the kernels use 32-bit and 24-bit arithmetic.
fq_status lis_constants(float s_logit, int32_t bits, int32_t n, int32_t Lk,
                        fqvit::LisConsts* k) {
    if (!(s_logit >= 1e-4f && s_logit <= 0.5f)) return FQ_ERR_PARAM;
    if (bits < 1 || bits > 8 || n < 1 || n > 30) return FQ_ERR_PARAM;
    const double s = (double)s_logit;
    const double q_ln2 = std::floor(-0.69314718055994530942 / s);   // floor(-ln2 / s)
    const double q_b = std::floor(1.353 / s);                       // floor(b / s)
    const double q_c = std::floor(0.344 / ((0.3585 * s) * s));      // floor(c / (a s^2))
    const uint64_t d = (uint64_t)(-q_ln2);
    const uint64_t qb = (uint64_t)q_b;
    const uint64_t qc = (uint64_t)q_c;
    // q_p + q_b lies in [q_b - d + 1, q_b]: positive and below 2^16; 3 q_L < 2^32.
    if (d < 1 || qb < d || qb >= 65536 || 3 * (qb * qb + qc) >= (1ull << 32)) return FQ_ERR_PARAM;
    int pre = 0;
    while ((d << pre) <= 256) ++pre;
    const uint64_t dp = d << pre;
    if ((uint64_t)n * dp * dp >= (1ull << 32) || (uint64_t)n * dp >= (1ull << 24)) return FQ_ERR_PARAM;
    // The row sum (and 2 sum + e) must stay below 2^63.
    const unsigned __int128 emax = (unsigned __int128)(qb * qb + qc) << n;
    if ((unsigned __int128)(2 * (uint64_t)Lk + 1) * emax >= ((unsigned __int128)1 << 63))
        return FQ_ERR_HEADROOM;
    k->d_ln2 = (uint32_t)d;
    k->qb = (uint32_t)qb;
    k->qc = (uint32_t)qc;
    k->u_max = (uint32_t)(n * d);
    k->magic = (uint32_t)((1ull << 32) / dp + 1);
    k->pre = pre;
    k->n = n;
    k->top = (1 << bits) - 1;
    // The float path: every e = qL 2^(n - z) is exact in binary32 (qL < 2^24)
    // and 2S + e stays below 2^52 (exact in binary64).
    const uint64_t qlmax = qb * qb + qc;
    k->fp_ok = qlmax < (1ull << 24) &&
               (unsigned __int128)(2 * (uint64_t)Lk + 1) * ((unsigned __int128)qlmax << n) <
                   ((unsigned __int128)1 << 52);
    return FQ_OK;
}

bool grid_fits(int64_t G, int32_t Lq, int32_t rows_per_block) {
    const int64_t tiles = (Lq + rows_per_block - 1) / rows_per_block;
    return G <= (int64_t)0x7FFFFFFF / (tiles > 0 ? tiles : 1);
}

}  // namespace

// Workspace of the calibration: the min/max partials, the per-block error sums
// of every candidate alpha and channel, and the per-channel totals.
size_t fqvit::ptf_calibrate_workspace_bytes(int64_t T, int32_t C, int32_t K) {
    const int64_t nb = (T + kPtfErrBlock - 1) / kPtfErrBlock;
    return (size_t)kMinmaxParts * 2 * sizeof(float) + (size_t)(K + 1) * nb * C * sizeof(double) +
           (size_t)(K + 1) * C * sizeof(double);
}

const fqvit::LaunchEvents& fqvit::launch_events() { return t_events; }
void fqvit::set_launch_events(hipEvent_t start, hipEvent_t stop) {
    t_events.start = start;
    t_events.stop = stop;
}

extern "C" {

const char* fq_status_str(int status) {
    switch (status) {
        case FQ_OK: return "FQ_OK";
        case FQ_ERR_NULL: return "FQ_ERR_NULL: a required pointer is NULL";
        case FQ_ERR_SHAPE: return "FQ_ERR_SHAPE: a size is out of the supported range";
        case FQ_ERR_PARAM: return "FQ_ERR_PARAM: a scalar parameter is out of range";
        case FQ_ERR_HEADROOM: return "FQ_ERR_HEADROOM: the i-exp row sum could overflow 64 bits";
        case FQ_ERR_HIP: return "FQ_ERR_HIP: the HIP runtime rejected a launch";
        case FQ_ERR_SCRATCH:
            return "FQ_ERR_SCRATCH: the call needs more than the library's fixed device scratch holds";
        default: return "unknown fq_status";
    }
}

int32_t fq_version(void) { return 100; }

fq_status fq_time_next_call(void* start_event, void* stop_event) {
    t_events.start = (hipEvent_t)start_event;
    t_events.stop = (hipEvent_t)stop_event;
    return FQ_OK;
}

fq_status ptf_layernorm_int8(const int8_t* x_q, int64_t T, int32_t C, int32_t zp_in,
                             const uint8_t* alpha, int32_t K, const float* gamma,
                             const float* beta, float s_out, int32_t zp_out, int32_t bits,
                             int8_t* y_q, void* stream) {
    ConsumeEvents consume;
    if (T < 0 || C < 1 || C > kMaxC) return FQ_ERR_SHAPE;
    if (bits < 2 || bits > 8 || K < 0 || K > 7) return FQ_ERR_PARAM;
    if (!(s_out > 0.0f) || !std::isfinite(s_out)) return FQ_ERR_PARAM;
    const int32_t half = 1 << (bits - 1);
    if (zp_in < -half || zp_in >= half || zp_out < -half || zp_out >= half) return FQ_ERR_PARAM;
    if (T == 0) return FQ_OK;
    if (!x_q || !alpha || !gamma || !beta || !y_q) return FQ_ERR_NULL;
    fqvit::LnArgs a{x_q, y_q, alpha, gamma, beta, T, C, zp_in, K, s_out, zp_out, bits};
    return from_hip(fqvit::launch_ptf_layernorm(a, (hipStream_t)stream));
}

fq_status lis_softmax_log4(const int32_t* logits, int64_t G, int32_t Lq, int32_t Lk,
                           const int32_t* bias, int32_t Hb, float s_logit, int32_t bits,
                           int32_t exp_n, uint8_t* codes, int32_t ld_codes, void* stream) {
    ConsumeEvents consume;
    // codes of up to 4 bits two per byte, wider codes one per byte
    const int32_t row_bytes = (bits >= 5 && bits <= 8) ? Lk : (Lk + 1) / 2;
    if (G < 0 || Lq < 0 || Lk < 1 || Lk > kMaxLk || ld_codes < row_bytes || (bias && Hb < 1) ||
        !grid_fits(G, Lq, 64))
        return FQ_ERR_SHAPE;
    fqvit::LisConsts k;
    const fq_status st = lis_constants(s_logit, bits, exp_n, Lk, &k);
    if (st != FQ_OK) return st;
    if (G == 0 || Lq == 0) return FQ_OK;
    if (!logits || !codes) return FQ_ERR_NULL;
    fqvit::LisArgs a{};
    a.logits = logits;
    a.bias = bias;
    a.Hb = bias ? Hb : 1;
    a.G = G;
    a.Lq = Lq;
    a.Lk = Lk;
    a.k = k;
    a.codes = codes;
    a.ld_codes = ld_codes;
    return from_hip(fqvit::launch_lis(a, (hipStream_t)stream));
}

fq_status lis_attn_v_shift(const uint8_t* codes, int32_t ld_codes, const int8_t* v,
                           int32_t zp_v, int64_t G, int32_t Lq, int32_t Lk, int32_t d,
                           int32_t bits, int32_t* out, void* stream) {
    ConsumeEvents consume;
    if (G < 0 || Lq < 0 || Lk < 1 || Lk > kMaxLk || d < 1 || d > kMaxD ||
        ld_codes < (Lk + 1) / 2 || !grid_fits(G, Lq, 16))
        return FQ_ERR_SHAPE;
    if (bits < 1 || bits > 4 || zp_v < -128 || zp_v > 127) return FQ_ERR_PARAM;
    if (G == 0 || Lq == 0) return FQ_OK;
    if (!codes || !v || !out) return FQ_ERR_NULL;
    fqvit::AvArgs a{codes, ld_codes, v, zp_v, G, Lq, Lk, d, (1 << bits) - 1, out};
    return from_hip(fqvit::launch_attn_v_shift(a, (hipStream_t)stream));
}

fq_status lis_attn_v_shift_wide(const uint8_t* codes, int32_t ld_codes, const int8_t* v,
                                int32_t zp_v, int64_t G, int32_t Lq, int32_t Lk, int32_t d,
                                int32_t bits, int64_t* out, void* stream) {
    ConsumeEvents consume;
    const int32_t row_bytes = (bits >= 5 && bits <= 8) ? Lk : (Lk + 1) / 2;
    if (G < 0 || Lq < 0 || Lk < 1 || Lk > kMaxLk || d < 1 || d > kMaxD || ld_codes < row_bytes ||
        !grid_fits(G, Lq, 16))
        return FQ_ERR_SHAPE;
    if (bits < 1 || bits > 8 || zp_v < -128 || zp_v > 127) return FQ_ERR_PARAM;
    if (G == 0 || Lq == 0) return FQ_OK;
    if (!codes || !v || !out) return FQ_ERR_NULL;
    const int32_t N = (1 << bits) - 1;
    fqvit::AvWideArgs a{codes, ld_codes, v, zp_v, G, Lq, Lk, d, bits, N < 44 ? N : 44, out};
    return from_hip(fqvit::launch_attn_v_shift_wide(a, (hipStream_t)stream));
}

fq_status lis_attention_head(const int32_t* logits, const int32_t* bias, int32_t Hb,
                             int64_t G, int32_t Lq, int32_t Lk, float s_logit, int32_t bits,
                             int32_t exp_n, const int8_t* v, int32_t zp_v, int32_t d,
                             int32_t* out, uint8_t* codes_out, int32_t ld_codes, void* stream) {
    ConsumeEvents consume;
    if (G < 0 || Lq < 0 || Lk < 1 || Lk > kMaxLk || d < 1 || d > kMaxD || (bias && Hb < 1) ||
        (codes_out && ld_codes < (Lk + 1) / 2) || !grid_fits(G, Lq, 64))
        return FQ_ERR_SHAPE;
    if (zp_v < -128 || zp_v > 127) return FQ_ERR_PARAM;
    if (bits > 4) return FQ_ERR_PARAM;   // the BitShift product shifts by at most 15
    fqvit::LisConsts k;
    const fq_status st = lis_constants(s_logit, bits, exp_n, Lk, &k);
    if (st != FQ_OK) return st;
    if (G == 0 || Lq == 0) return FQ_OK;
    if (!logits || !v || !out) return FQ_ERR_NULL;
    fqvit::LisArgs a{};
    a.logits = logits;
    a.bias = bias;
    a.Hb = bias ? Hb : 1;
    a.G = G;
    a.Lq = Lq;
    a.Lk = Lk;
    a.k = k;
    a.v = v;
    a.zp_v = zp_v;
    a.d = d;
    a.out = out;
    a.codes = codes_out;
    a.ld_codes = codes_out ? ld_codes : 0;
    return from_hip(fqvit::launch_lis(a, (hipStream_t)stream));
}

fq_status lis_attention_qk(const int8_t* q, const int8_t* k, int32_t zp_q, int32_t zp_k,
                           int32_t dk, const int32_t* bias, int32_t Hb, int64_t G, int32_t Lq,
                           int32_t Lk, float s_logit, int32_t bits, int32_t exp_n,
                           const int8_t* v, int32_t zp_v, int32_t d, int32_t* out, void* stream) {
    ConsumeEvents consume;
    if (G < 0 || G > 0x7FFFFFFF || Lq < 0 || Lk < 1 || Lk > fqvit::kQkMaxLk || d < 1 || d > 64 ||
        (dk != 32 && dk != 64) || (bias && Hb < 1))
        return FQ_ERR_SHAPE;
    if (zp_q < -128 || zp_q > 127 || zp_k < -128 || zp_k > 127 || zp_v < -128 || zp_v > 127)
        return FQ_ERR_PARAM;
    if (bits > 4) return FQ_ERR_PARAM;   // the BitShift product shifts by at most 15
    fqvit::LisConsts kc;
    const fq_status st = lis_constants(s_logit, bits, exp_n, Lk, &kc);
    if (st != FQ_OK) return st;
    if (G == 0 || Lq == 0) return FQ_OK;
    if (!q || !k || !v || !out) return FQ_ERR_NULL;
    if (((reinterpret_cast<uintptr_t>(q) | reinterpret_cast<uintptr_t>(k)) & 15) != 0)
        return FQ_ERR_PARAM;
    fqvit::LisArgs a{};
    a.bias = bias;
    a.Hb = bias ? Hb : 1;
    a.G = G;
    a.Lq = Lq;
    a.Lk = Lk;
    a.k = kc;
    a.v = v;
    a.zp_v = zp_v;
    a.d = d;
    a.out = out;
    const fqvit::QkInput in{q, k, zp_q, zp_k, dk};
    return from_hip(fqvit::launch_lis_qk(a, in, (hipStream_t)stream));
}

size_t fq_ptf_calibrate_workspace_bytes(int64_t T, int32_t C, int32_t K) {
    if (T < 1 || T > kMaxCalibT || C < 1 || C > kMaxC || K < 0 || K > 7) return 0;
    return fqvit::ptf_calibrate_workspace_bytes(T, C, K);
}

fq_status ptf_calibrate(const float* x, int64_t T, int32_t C, int32_t bits, int32_t K, double* s,
                        int32_t* zp, uint8_t* alpha, void* workspace, size_t workspace_bytes,
                        void* stream) {
    ConsumeEvents consume;
    if (T < 0 || T > kMaxCalibT || C < 1 || C > kMaxC) return FQ_ERR_SHAPE;
    if (bits < 2 || bits > 8 || K < 0 || K > 7) return FQ_ERR_PARAM;
    if (T == 0) return FQ_OK;
    if (!x || !s || !zp || !alpha || !workspace) return FQ_ERR_NULL;
    if (workspace_bytes < fqvit::ptf_calibrate_workspace_bytes(T, C, K)) return FQ_ERR_PARAM;
    fqvit::PtfCalibArgs a{x, T, C, bits, K, s, zp, alpha, workspace};
    return from_hip(fqvit::launch_ptf_calibrate(a, (hipStream_t)stream));
}

fq_status ptf_calibrate_noalloc(const float* x, int64_t T, int32_t C, int32_t bits, int32_t K,
                                double* s, int32_t* zp, uint8_t* alpha, void* stream) {
    ConsumeEvents consume;
    if (T < 0 || T > kMaxCalibT || C < 1 || C > kMaxC) return FQ_ERR_SHAPE;
    if (bits < 2 || bits > 8 || K < 0 || K > 7) return FQ_ERR_PARAM;
    if (T == 0) return FQ_OK;
    if (!x || !s || !zp || !alpha) return FQ_ERR_NULL;
    if (fqvit::ptf_calibrate_workspace_bytes(T, C, K) > FQ_NOALLOC_SCRATCH_BYTES)
        return FQ_ERR_SCRATCH;
    fqvit::PtfCalibArgs a{x, T, C, bits, K, s, zp, alpha, nullptr};
    return from_hip(fqvit::launch_ptf_calibrate_noalloc(a, (hipStream_t)stream));
}

fq_status ptf_quantize_int8(const float* x, int64_t T, int32_t C, const double* s,
                            const int32_t* zp, const uint8_t* alpha, int32_t bits, int8_t* x_q,
                            void* stream) {
    ConsumeEvents consume;
    if (T < 0 || C < 1 || C > kMaxC) return FQ_ERR_SHAPE;
    if (bits < 2 || bits > 8) return FQ_ERR_PARAM;
    if (T == 0) return FQ_OK;
    if (!x || !s || !zp || !alpha || !x_q) return FQ_ERR_NULL;
    fqvit::PtfQuantArgs a{x, T, C, s, zp, alpha, bits, x_q};
    return from_hip(fqvit::launch_ptf_quantize(a, (hipStream_t)stream));
}

fq_status requant_dyadic_int8(const int32_t* q, int64_t n, float s_in, float s_out,
                              int32_t zp_out, int32_t bits, int8_t* y, void* stream) {
    ConsumeEvents consume;
    if (n < 0) return FQ_ERR_SHAPE;
    if (bits < 2 || bits > 8) return FQ_ERR_PARAM;
    if (!(s_in > 0.0f) || !std::isfinite(s_in) || !(s_out > 0.0f) || !std::isfinite(s_out))
        return FQ_ERR_PARAM;
    const int32_t half = 1 << (bits - 1);
    if (zp_out < -half || zp_out >= half) return FQ_ERR_PARAM;
    if (n == 0) return FQ_OK;
    if (!q || !y) return FQ_ERR_NULL;
    // N2 / 2^N1: the 31-bit dyadic form of M = s_in / s_out.
    const double M = (double)s_in / (double)s_out;
    int e = 0;
    (void)std::frexp(M, &e);
    int64_t N1 = 31 - (int64_t)e;
    N1 = N1 < 0 ? 0 : (N1 > 62 ? 62 : N1);
    double n2 = std::floor(std::ldexp(M, (int)N1));
    if (n2 > 2147483647.0) n2 = 2147483647.0;
    fqvit::RequantArgs a{q, n, (int64_t)n2, (int32_t)N1, zp_out, bits, y};
    return from_hip(fqvit::launch_requant(a, (hipStream_t)stream));
}

}  // extern "C"
