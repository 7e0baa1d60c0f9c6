// Internal declarations shared by the gfx950 kernels and the C ABI wrappers of
// libfqvit.  Not part of the public interface (include/fqvit.h is).  Only the
// HIP runtime API types are needed here, so the C ABI's host code compiles with
// any C++17 compiler; the launch helper lives in fqvit_launch.h.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace fqvit {

// Events attached to the kernel of the current entry-point call on this thread
// (set by fq_time_next_call, cleared when that call returns).
struct LaunchEvents {
    hipEvent_t start = nullptr;
    hipEvent_t stop = nullptr;
};
const LaunchEvents& launch_events();
// Replaces the current call's events (for entry points that launch several
// kernels: the start event goes on the first, the stop event on the last).
void set_launch_events(hipEvent_t start, hipEvent_t stop);

// ---------------------------------------------------------------------------
// PTF LayerNorm
// ---------------------------------------------------------------------------

struct LnArgs {
    const int8_t* x;
    int8_t* y;
    const uint8_t* alpha;
    const float* gamma;
    const float* beta;
    int64_t T;
    int32_t C;
    int32_t zp_in;     // container form
    int32_t K;
    float s_out;
    int32_t zp_out;    // container form
    int32_t bits;
};

hipError_t launch_ptf_layernorm(const LnArgs& a, hipStream_t stream);

// ---------------------------------------------------------------------------
// Log-Int-Softmax / BitShift attention
// ---------------------------------------------------------------------------

// Integer constants of the I-Exp / code pipeline, derived on the host.
struct LisConsts {
    uint32_t d_ln2;     // -q_ln2 = -floor(-ln2 / s) > 0
    uint32_t qb;        // floor(1.353 / s)
    uint32_t qc;        // floor(0.344 / ((0.3585 s) s))
    uint32_t u_max;     // n * d_ln2: inputs below -u_max are clamped
    uint32_t magic;     // floor(2^32 / (d_ln2 << pre)) + 1
    int32_t pre;        // pre-shift making (d_ln2 << pre) > 256
    int32_t n;          // clamp depth
    int32_t top;        // 2^bits - 1
    // The float path (e held exactly in binary32, the row sum and the code's
    // values exactly in binary64) is valid when q_b^2 + q_c < 2^24 and
    // (2 Lk + 1)(q_b^2 + q_c) 2^n < 2^52.
    int32_t fp_ok;
};

struct LisArgs {
    const int32_t* logits;  // [G, Lq, Lk]
    const int32_t* bias;    // nullable [Hb, Lq, Lk]
    int32_t Hb;
    int64_t G;
    int32_t Lq, Lk;
    LisConsts k;
    // fused / A.V part
    const int8_t* v;        // [G, Lk, d]  (nullable for codes-only)
    int32_t zp_v;
    int32_t d;
    int32_t* out;           // [G, Lq, d]  (nullable for codes-only)
    uint8_t* codes;         // nullable [G, Lq, ld_codes]
    int32_t ld_codes;
};

hipError_t launch_lis(const LisArgs& a, hipStream_t stream);

// Integer-only attention from int8 Q and K (logits computed on chip; the
// logits / codes fields of LisArgs are unused).
struct QkInput {
    const int8_t* q;        // [G, Lq, dk]
    const int8_t* k;        // [G, Lk, dk]
    int32_t zp_q, zp_k;     // container form
    int32_t dk;             // 32 or 64
};

constexpr int kQkMaxLk = 640;   // keys per unit (20 chunks of 32)

hipError_t launch_lis_qk(const LisArgs& a, const QkInput& in, hipStream_t stream);

struct AvArgs {
    const uint8_t* codes;
    int32_t ld_codes;
    const int8_t* v;
    int32_t zp_v;
    int64_t G;
    int32_t Lq, Lk, d;
    int32_t top;            // 2^bits - 1
    int32_t* out;
};

hipError_t launch_attn_v_shift(const AvArgs& a, hipStream_t stream);

// The same product on the int8 matrix cores (rows of up to kAvMfmaMaxLk keys,
// d <= 64); hipErrorNotSupported for other shapes.  AvMfma: its launch
// parameters (both products).
constexpr int kAvMfmaMaxLk = 1024;
struct AvMfma {
    uint32_t lut[3][4];   // P_k bytes for codes 0..15, four per dword
    int kp;               // keys padded to a multiple of 64
    int nks;              // kp / 64
    int ldv;              // LDS row stride of V^T in bytes (kp + 16)
    int ntiles;           // 16-row tiles per unit
    int unit_bytes;       // code bytes a unit spans: (Lq - 1) ld_codes + ceil(Lk / 2)
    int vec_out;          // 16-byte output stores (d % 4 == 0, 16-byte aligned out)
    int vec_v;            // V rows read as 16-byte units (d % 16 == 0, 16-byte aligned V)
};
hipError_t launch_attn_v_mfma(const AvArgs& a, hipStream_t stream);

// BitShift product for codes of any width: int64 output at scale s_V / 2^W.
struct AvWideArgs {
    const uint8_t* codes;
    int32_t ld_codes;
    const int8_t* v;
    int32_t zp_v;
    int64_t G;
    int32_t Lq, Lk, d;
    int32_t bits;           // code width: nibbles for <= 4, bytes above
    int32_t W;              // output exponent min(2^bits - 1, 44)
    int64_t* out;
};

hipError_t launch_attn_v_shift_wide(const AvWideArgs& a, hipStream_t stream);
// The wide product on the int8 matrix cores (same shape limits as
// launch_attn_v_mfma); hipErrorNotSupported for other shapes.
hipError_t launch_attn_v_wide_mfma(const AvWideArgs& a, hipStream_t stream);

// ---------------------------------------------------------------------------
// PTF calibration / quantization and dyadic requantization
// ---------------------------------------------------------------------------

constexpr int kPtfErrBlock = 64;     // rows per block of the alpha-search error sums
constexpr int kMinmaxParts = 1024;   // at most this many min/max partials

struct PtfCalibArgs {
    const float* x;         // [T, C]
    int64_t T;
    int32_t C, bits, K;
    double* s;              // device scalar out
    int32_t* zp;            // device scalar out (container form)
    uint8_t* alpha;         // [C] out
    void* workspace;        // ptf_calibrate_workspace_bytes(T, C, K) bytes
};

size_t ptf_calibrate_workspace_bytes(int64_t T, int32_t C, int32_t K);
hipError_t launch_ptf_calibrate(const PtfCalibArgs& a, hipStream_t stream);
// The same with the workspace in the library's fixed device array (the
// caller has checked the size against FQ_NOALLOC_SCRATCH_BYTES; a.workspace
// is ignored).
hipError_t launch_ptf_calibrate_noalloc(const PtfCalibArgs& a, hipStream_t stream);

struct PtfQuantArgs {
    const float* x;         // [T, C]
    int64_t T;
    int32_t C;
    const double* s;        // device scalar
    const int32_t* zp;      // device scalar (container form)
    const uint8_t* alpha;   // [C]
    int32_t bits;
    int8_t* y;              // [T, C]
};

hipError_t launch_ptf_quantize(const PtfQuantArgs& a, hipStream_t stream);

struct RequantArgs {
    const int32_t* q;
    int64_t n;
    int64_t N2;             // in [0, 2^31 - 1]
    int32_t N1;             // in [0, 62]
    int32_t zp;             // container form
    int32_t bits;
    int8_t* y;
};

hipError_t launch_requant(const RequantArgs& a, hipStream_t stream);

}  // namespace fqvit
