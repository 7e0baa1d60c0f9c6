// Device code of the Log-Int-Softmax attention kernels for gfx950 (Supplement A.2: Algorithm 1 I-Exp,
// Algorithm 2 I-Log2 and Log-Int-Softmax, the clip of the LIS equation; the
// BitShift product with V of Sec. 3.3 and its zero-point form).
//
// Lane layout.  A wavefront owns 16 query rows of one attention unit g
// (image x window x head).  Lane (r, kg) = (lane % 16, lane / 16) holds row r
// and, in every 32-key chunk c, the eight keys
//     32c + 4kg + t       (t = 0..3)   and   32c + 16 + 4kg + t   (t = 0..3),
// so each 16-byte load of a lane is contiguous and the four lanes of a row
// cover 64 contiguous bytes per load instruction.  The same eight keys are the
// eight k-slots the lane feeds to the 16x16x32 bf16 MFMA (the first four are
// its k-slots of the 16x16x16 MFMA used for a last chunk of at most 16 keys);
// V^T is staged in LDS with its keys permuted the same way, so the contraction
// pairs every key of the attention row with its own V row.
//
// Per row: max (lane-local, then two cross-lane shuffles), I-Exp and the exact
// sum S, then the code of every key.  The codes never leave the chip in the
// fused kernels: each becomes P = 2^(N - code) as a bf16 bit pattern and the
// chunk is multiplied with V^T by MFMA.  That product is exact: P and V - zp_V
// are exact in bf16, every product is an integer and every partial sum is an
// integer of magnitude below 2^24 (the codes of a row satisfy
// sum_j 2^-code_j < 1.5 + (Lk - 1)/2^15, so |out| < 255 (1.5 2^15 + Lk) < 2^24
// for Lk <= 4096), so fp32 accumulation in any order rounds nothing.
//
// The code needs no division.  With e = qL 2^s (qL = (q_p + q_b)^2 + q_c,
// s = n - z) and r = round(S / e) (ties up), I-Log2(r) >= k exactly when
// 2S >= c_k e with c_1 = 3 and c_k = 3 2^(k-1) - 1: for k >= 2 that is
// (2S + e) / (1.5 e) >= 2^k, and for k = 1 it is 2S >= 3e.  Hence
//     code = min(m, N) - [2S < 3e],   m = floor(log2((2S + e) / (1.5 e))),
// (m >= 1 always, since 2S >= 2e, and 2S < 3e forces m = 1).  Two exact
// evaluations of this formula are implemented:
//   * float path: I-Exp by the 24-bit integer steps, e = qL 2^(n - z) held as
//     a binary32 value (qL < 2^24), the row sum in binary64, and the code
//     from binary64 values (2S + e below 2^52), m being the
//     difference of the IEEE bit patterns of 2S + e and 1.5 e shifted right
//     by 52 (both positive, so the pattern difference is the exponent
//     difference minus a borrow exactly when the significand of the quotient
//     falls below 1), taken on the patterns shifted right by 27 so that it is
//     32-bit arithmetic, and [2S < 3e] a binary32 comparison of e with
//     floor(2S / 3);
//   * integer path (any scale the host accepts): 24-bit integer I-Exp and
//     64-bit comparisons.  With Sp = floor(2S / 2^s), W = Sp + qL and Q = 3 qL,
//     m = floor(log2(W / Q)) + 1 and 2S < 3e is Sp < Q; msb(W) is msb(2S) - s
//     or one more, so floor(log2(W / Q)) is j0 - 1, j0 or j0 + 1 with
//     j0 = msb(2S) - s - msb(Q), settled by two comparisons.
// The host picks the float path whenever its exactness conditions hold.
#pragma once

#include "fqvit_launch.h"

namespace fqvit {
namespace lis {

constexpr int kBlock = 256;        // four wavefronts
constexpr int kRowsPerBlock = 64;  // 16 rows per wavefront in the tile kernel

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int32_t i32x4a4 __attribute__((ext_vector_type(4), aligned(4)));

// Block index -> logical tile so that the tiles of one unit run on one XCD
// (blocks are dealt round-robin to the eight XCDs) and share its L2.
__device__ __forceinline__ int64_t xcd_remap(int64_t b, int64_t total) {
    const int64_t per = total >> 3;
    if (b >= (per << 3)) return b;
    return (b & 7) * per + (b >> 3);
}

// Position of key j (0..31) of a chunk in the permuted order: the eight keys
// of lane group kg are contiguous.
__device__ __forceinline__ int chunk_pos(int j) {
    return ((j & 15) >> 2) * 8 + ((j >> 4) << 2) + (j & 3);
}

// ---------------------------------------------------------------------------
// Reductions over the four lanes of a row (l, l ^ 16, l ^ 32, l ^ 48) with the
// lane-swap instructions (v_permlane32_swap, v_permlane16_swap): they stay in
// the VALU, where a shuffle would take an LDS round trip.  Swapping a value
// with itself leaves, per lane, the value of lane l and of its partner in the
// two results.  The whole wavefront must be active.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int row4_max(int v) {
    const auto s = __builtin_amdgcn_permlane32_swap((uint32_t)v, (uint32_t)v, false, false);
    v = max((int)s[0], (int)s[1]);
    const auto t = __builtin_amdgcn_permlane16_swap((uint32_t)v, (uint32_t)v, false, false);
    return max((int)t[0], (int)t[1]);
}

__device__ __forceinline__ int row4_sum(int v) {
    const auto s = __builtin_amdgcn_permlane32_swap((uint32_t)v, (uint32_t)v, false, false);
    v = (int)(s[0] + s[1]);
    const auto t = __builtin_amdgcn_permlane16_swap((uint32_t)v, (uint32_t)v, false, false);
    return (int)(t[0] + t[1]);
}

__device__ __forceinline__ uint64_t row4_sum(uint64_t v) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
        const auto sl = h == 0 ? __builtin_amdgcn_permlane32_swap(lo, lo, false, false)
                               : __builtin_amdgcn_permlane16_swap(lo, lo, false, false);
        const auto sh = h == 0 ? __builtin_amdgcn_permlane32_swap(hi, hi, false, false)
                               : __builtin_amdgcn_permlane16_swap(hi, hi, false, false);
        v = (((uint64_t)sh[0] << 32) | sl[0]) + (((uint64_t)sh[1] << 32) | sl[1]);
    }
    return v;
}

// Exact when every partial sum is (integers below 2^53 here).
__device__ __forceinline__ double row4_sum(double v) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const uint64_t b = (uint64_t)__double_as_longlong(v);
        const uint32_t lo = (uint32_t)b, hi = (uint32_t)(b >> 32);
        const auto sl = h == 0 ? __builtin_amdgcn_permlane32_swap(lo, lo, false, false)
                               : __builtin_amdgcn_permlane16_swap(lo, lo, false, false);
        const auto sh = h == 0 ? __builtin_amdgcn_permlane32_swap(hi, hi, false, false)
                               : __builtin_amdgcn_permlane16_swap(hi, hi, false, false);
        v = __longlong_as_double((int64_t)(((uint64_t)sh[0] << 32) | sl[0])) +
            __longlong_as_double((int64_t)(((uint64_t)sh[1] << 32) | sl[1]));
    }
    return v;
}

// ---------------------------------------------------------------------------
// V^T staging.  Keys [k0, k0 + kcnt) of V[g] go to vt[col][pos] as bf16 bits of
// v - zp (kcnt a multiple of 32).  A work item is four consecutive keys (one
// 8-byte run of the permuted order) and 16 columns: four 16-byte loads, then
// per column two bf16 pairs written with one 8-byte LDS store.  Consecutive
// threads take consecutive key quads, so a wavefront's stores to one column
// row are contiguous.  Conversion: the byte b of v is flipped to b ^ 0x80
// (= v + 128, unsigned), converted to float and reduced by 128 + zp, which is
// exact; the bf16 pattern is the high half of that float.  Keys past Lk and
// columns past d hold -zp: those keys get P = 0 and those columns are never
// stored, so any finite value is harmless.
// ---------------------------------------------------------------------------
constexpr int kStageItems = 2;     // items per thread and stage: kcnt dpad / 64 <= 512

struct StageRegs {
    u32x4 w[kStageItems][4];
};

__device__ __forceinline__ u32x4 load_v16(const int8_t* vrow, int dd, int d, bool vec_ok) {
    if (vec_ok) return *reinterpret_cast<const u32x4*>(vrow + dd);
    u32x4 w = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int q = 0; q < 16; ++q)
        if (dd + q < d) w[q >> 2] |= (uint32_t)(uint8_t)vrow[dd + q] << (8 * (q & 3));
    return w;
}

template <int NTHREADS = kBlock>
__device__ __forceinline__ void stage_load(StageRegs& sr, const int8_t* vg, int Lk, int d,
                                           int ncg, int k0, int kcnt, bool vec_ok) {
    const int nquads = kcnt >> 2;
    const int nitems = nquads * ncg;
#pragma unroll
    for (int it = 0; it < kStageItems; ++it) {
        const int idx = (int)threadIdx.x + it * NTHREADS;
        const int cg = idx / nquads;
        const int j = k0 + 4 * (idx - cg * nquads);
        const int dd = 16 * cg;
        const bool ok = idx < nitems && dd < d;
#pragma unroll
        for (int t = 0; t < 4; ++t)
            sr.w[it][t] = (ok && j + t < Lk) ? load_v16(vg + (int64_t)(j + t) * d, dd, d, vec_ok)
                                             : u32x4{0u, 0u, 0u, 0u};
    }
}

// Two bf16 from the high halves of two floats: lo in bits 0..15, hi in 16..31.
__device__ __forceinline__ uint32_t bf16_pair(float lo, float hi) {
    return __builtin_amdgcn_perm(__float_as_uint(hi), __float_as_uint(lo), 0x07060302u);
}

template <int NTHREADS = kBlock>
__device__ __forceinline__ void stage_store(const StageRegs& sr, uint16_t* vt, int ld, int ncg,
                                            int kcnt, int zp) {
    const int nquads = kcnt >> 2;
    const int nitems = nquads * ncg;
    const float off = (float)(128 + zp);
#pragma unroll
    for (int it = 0; it < kStageItems; ++it) {
        const int idx = (int)threadIdx.x + it * NTHREADS;
        if (idx >= nitems) continue;
        const int cg = idx / nquads;
        const int jj = 4 * (idx - cg * nquads);
        const int pos = (jj & ~31) + chunk_pos(jj & 31);
        u32x4 w[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) w[t] = sr.w[it][t] ^ 0x80808080u;
#pragma unroll
        for (int q = 0; q < 16; ++q) {
            float f[4];
#pragma unroll
            for (int t = 0; t < 4; ++t)
                f[t] = (float)((w[t][q >> 2] >> (8 * (q & 3))) & 0xFFu) - off;
            *reinterpret_cast<u32x2*>(vt + (16 * cg + q) * ld + pos) =
                u32x2{bf16_pair(f[0], f[1]), bf16_pair(f[2], f[3])};
        }
    }
}

// Staging of one V^T stage by the whole workgroup.
__device__ __forceinline__ void stage_vt(uint16_t* vt, int ld, const int8_t* vg, int Lk, int d,
                                         int ncg, int k0, int kcnt, int zp, bool vec_ok) {
    StageRegs sr;
    stage_load(sr, vg, Lk, d, ncg, k0, kcnt, vec_ok);
    stage_store(sr, vt, ld, ncg, kcnt, zp);
}

// ---------------------------------------------------------------------------
// Logits
// ---------------------------------------------------------------------------

// Load the 8 logits (+ bias) of lane (r, kg) in a chunk whose 32 keys are all valid.
__device__ __forceinline__ void load_full(int (&dst)[8], const int32_t* row, const int32_t* brow,
                                          int c, int kg) {
    const int k0 = 32 * c + 4 * kg;
    const i32x4a4 a = *reinterpret_cast<const i32x4a4*>(row + k0);
    const i32x4a4 b = *reinterpret_cast<const i32x4a4*>(row + k0 + 16);
    dst[0] = a.x; dst[1] = a.y; dst[2] = a.z; dst[3] = a.w;
    dst[4] = b.x; dst[5] = b.y; dst[6] = b.z; dst[7] = b.w;
    if (brow) {
        const i32x4a4 ba = *reinterpret_cast<const i32x4a4*>(brow + k0);
        const i32x4a4 bb = *reinterpret_cast<const i32x4a4*>(brow + k0 + 16);
        dst[0] += ba.x; dst[1] += ba.y; dst[2] += ba.z; dst[3] += ba.w;
        dst[4] += bb.x; dst[5] += bb.y; dst[6] += bb.z; dst[7] += bb.w;
    }
}

// Load the 8 logits (+ bias) of lane (r, kg) in chunk c; keys past Lk get
// INT_MIN.  vec_ok: the row and bias row are followed by at least 32 * (c + 1)
// readable elements inside their tensors, so the chunk is read with full
// vectors and masked afterwards.  HALF: only the first four keys (the last
// chunk holds at most 16 keys).
// DEFER: keys past Lk read with full vectors are left as loaded, to be masked
// by mask_last when the chunk is used; masking them here would make the
// wavefront wait for the load (and every load before it) right away.
template <bool HALF, bool DEFER = false>
__device__ __forceinline__ void load_chunk(int (&dst)[8], const int32_t* row, const int32_t* brow,
                                           int c, int kg, int Lk, bool vec_ok) {
    const int k0 = 32 * c + 4 * kg;
    const int k1 = k0 + 16;
    if (HALF) {
        if (vec_ok || k0 + 4 <= Lk) {
            const i32x4a4 a = *reinterpret_cast<const i32x4a4*>(row + k0);
            dst[0] = a.x; dst[1] = a.y; dst[2] = a.z; dst[3] = a.w;
            if (brow) {
                const i32x4a4 ba = *reinterpret_cast<const i32x4a4*>(brow + k0);
                dst[0] += ba.x; dst[1] += ba.y; dst[2] += ba.z; dst[3] += ba.w;
            }
            if (!DEFER) {
#pragma unroll
                for (int t = 0; t < 4; ++t)
                    if (k0 + t >= Lk) dst[t] = INT_MIN;
            }
        } else {
#pragma unroll
            for (int t = 0; t < 4; ++t)
                dst[t] = k0 + t < Lk ? row[k0 + t] + (brow ? brow[k0 + t] : 0) : INT_MIN;
        }
#pragma unroll
        for (int t = 4; t < 8; ++t) dst[t] = INT_MIN;
        return;
    }
    if (vec_ok || k1 + 4 <= Lk) {
        load_full(dst, row, brow, c, kg);
        if (!DEFER) {
#pragma unroll
            for (int t = 0; t < 8; ++t) {
                const int key = (t < 4 ? k0 : k1 - 4) + t;
                if (key >= Lk) dst[t] = INT_MIN;
            }
        }
    } else {
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            const int key = (t < 4 ? k0 : k1 - 4) + t;
            dst[t] = key < Lk ? row[key] + (brow ? brow[key] : 0) : INT_MIN;
        }
    }
}

// Valid keys of lane kg in the last chunk c = NC - 1, bit t for its key t.
template <int NC>
__device__ __forceinline__ uint32_t last_valid(int kg, int Lk) {
    const int k0 = 32 * (NC - 1) + 4 * kg;
    uint32_t m = 0;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
        const int key = (t < 4 ? k0 : k0 + 12) + t;
        m |= key < Lk ? 1u << t : 0u;
    }
    return m;
}

// The masking deferred by load_chunk<HALF, true>: keys past Lk of the last
// chunk become INT_MIN.
template <int NC, int NT>
__device__ __forceinline__ void mask_last(int (&lg)[NC][8], uint32_t valid) {
#pragma unroll
    for (int t = 0; t < NT; ++t) lg[NC - 1][t] = (valid >> t) & 1u ? lg[NC - 1][t] : INT_MIN;
}

// Store the 8 codes of lane (r, kg) in chunk c as nibbles (even key low).
__device__ __forceinline__ void store_codes(uint8_t* crow, int nbytes, int c, int kg,
                                            const int (&code)[8]) {
    const int b0 = 16 * c + 2 * kg;
    const int b1 = b0 + 8;
    const uint8_t v0 = (uint8_t)(code[0] | (code[1] << 4));
    const uint8_t v1 = (uint8_t)(code[2] | (code[3] << 4));
    const uint8_t v2 = (uint8_t)(code[4] | (code[5] << 4));
    const uint8_t v3 = (uint8_t)(code[6] | (code[7] << 4));
    if (b0 < nbytes) crow[b0] = v0;
    if (b0 + 1 < nbytes) crow[b0 + 1] = v1;
    if (b1 < nbytes) crow[b1] = v2;
    if (b1 + 1 < nbytes) crow[b1 + 1] = v3;
}

// Store the 8 codes of lane (r, kg) in chunk c of a row: nibbles for codes of
// up to 4 bits (top <= 15), else one byte per code (keys past Lk skipped).
__device__ __forceinline__ void store_codes_row(uint8_t* crow, int Lk, int top, int c, int kg,
                                                const int (&code)[8]) {
    if (top > 15) {
        const int k0 = 32 * c + 4 * kg;
#pragma unroll
        for (int t = 0; t < 4; ++t)
            if (k0 + t < Lk) crow[k0 + t] = (uint8_t)code[t];
#pragma unroll
        for (int t = 0; t < 4; ++t)
            if (k0 + 16 + t < Lk) crow[k0 + 16 + t] = (uint8_t)code[4 + t];
    } else {
        store_codes(crow, (Lk + 1) >> 1, c, kg, code);
    }
}

// Keys of V^T per LDS stage for a padded head dimension dpad: at most 40 KB of
// LDS per workgroup so that several workgroups share a CU.
constexpr int vt_stage_keys(int dpad) { return (40960 / (2 * dpad) - 8) / 32 * 32; }

struct LisLaunch {
    int ntiles;     // tile kernel: row tiles of 64 per unit; unit kernel: 16-row tiles per unit
    int kb;         // keys per V^T stage (multiple of 32)
    int ld;         // LDS row stride of V^T in bf16 elements
    int dpad;       // 16 * (power of two >= ceil(d / 16))
    int ncg;        // dpad / 16: 16-column groups of V
    int vec_ok;     // V rows read as 16-byte vectors (d % 16 == 0, 16-byte aligned V)
    int vt_bytes;   // LDS bytes of one V^T stage (0 for codes only)
    int out_vec;    // output rows written through LDS as 16-byte units (d % 4 == 0, aligned out)
    int64_t n_logits;  // elements of the logits tensor (G Lq Lk)
    int64_t n_bias;    // elements of the bias tensor (Hb Lq Lk), 0 without bias
    int tab_bytes;     // long-row kernel: LDS bytes of the I-Exp table (multiple of 16)
    int codes_ldw;     // unit kernel, codes only: LDS bytes per wavefront of the tile's
                       // code rows (dense rows, ld_codes = row bytes), 0: direct stores
};

// ---------------------------------------------------------------------------
// Integer path
// ---------------------------------------------------------------------------

// Per-row state after the I-Exp pass.
struct RowSum {
    uint64_t S2;    // 2 * sum_j e_j
    int rc;         // msb(S2) - 31 - n: j0 = rc + z + clz(3 qL)
};

__device__ __forceinline__ RowSum row_sum(uint64_t sum, const LisConsts& k) {
    sum = row4_sum(sum);
    RowSum rs;
    rs.S2 = sum << 1;
    rs.rc = (63 - __clzll((long long)rs.S2)) - 31 - k.n;
    return rs;
}

// I-Exp of one key (Algorithm 1): returns qL = (q_p + q_b)^2 + q_c and z; the
// i-exp value is e = qL << (n - z).  u = -q clamped to n * d_ln2; z = floor(u
// / d_ln2) by a 24-bit multiply-high with magic = floor(2^32 / (d << pre)) + 1,
// exact for u <= n d with n (d << pre)^2 < 2^32 and (d << pre) > 256.
__device__ __forceinline__ uint32_t iexp_qL(int v, int mx, const LisConsts& k, uint32_t& z) {
    const uint32_t u = min((uint32_t)mx - (uint32_t)v, k.u_max);
    z = (uint32_t)(((uint64_t)((u << k.pre) & 0xFFFFFFu) * (uint64_t)k.magic) >> 32);
    const uint32_t w = (k.qb - u + __umul24(z, k.d_ln2)) & 0xFFFFu;            // q_p + q_b
    return __umul24(w, w) + k.qc;
}

// Code min(I-Log2(round(S / e)), N) of one key from its qL, z and the row state.
__device__ __forceinline__ int lis_code(uint32_t qL, uint32_t z, const RowSum& rs,
                                         const LisConsts& k) {
    const uint64_t Sp = rs.S2 >> (k.n - (int)z);
    const uint64_t W = Sp + qL;
    const uint32_t Q = qL + (qL << 1);
    const int j0 = max(rs.rc + (int)z + (int)__builtin_clz(Q), 0);
    const uint64_t QJ = (uint64_t)Q << j0;
    const int code = j0 + (W >= QJ ? 1 : 0) + (W >= (QJ << 1) ? 1 : 0) - (Sp < (uint64_t)Q ? 1 : 0);
    return min(code, k.top);
}

// ---------------------------------------------------------------------------
// Float path
// ---------------------------------------------------------------------------

// I-Exp of one key for the float path, from its clamped input u = max - v:
// e = qL 2^(n - z) as a binary32 value (exact: qL < 2^24).  z, q_p + q_b and qL
// come from the 24-bit integer
// steps of iexp_qL (magic division by a multiply-high, two 24-bit
// multiply-adds), which cost less than binary32 arithmetic; the host accepts
// only scales for which those steps are exact.  k.magic and the shifted u are
// below 2^24, so the product maps to one v_mul_hi_u32_u24.
// P0: the pre-shift is known to be 0 (|q_ln2| > 256, i.e. s below about
// 2.7e-3), which saves the shift of every key.
template <bool P0 = false>
__device__ __forceinline__ float iexp_fu(uint32_t u, const LisConsts& k) {
    const uint32_t us = P0 ? u : (u << k.pre);
    const uint32_t z =
        (uint32_t)(((uint64_t)(us & 0xFFFFFFu) * (uint64_t)(k.magic & 0xFFFFFFu)) >> 32);
    // q_p + q_b = z d + (q_b - u); written out because the compiler would
    // otherwise select a 64-bit multiply-add
    uint32_t w;
    asm("v_mad_u32_u24 %0, %1, %2, %3" : "=v"(w) : "v"(z), "s"(k.d_ln2), "v"(k.qb - u));
    const uint32_t qL = __umul24(w, w) + k.qc;
    return __builtin_ldexpf((float)qL, k.n - (int)z);
}

// The same for a logit v of a row with maximum mx: u = mx - v clamped at
// n |q_ln2|.
template <bool P0 = false>
__device__ __forceinline__ float iexp_f(int v, int mx, const LisConsts& k) {
    return iexp_fu<P0>(min((uint32_t)mx - (uint32_t)v, k.u_max), k);
}

// Code of one key on the float path, from e (its binary32 bit pattern) and the
// row state (2S < 2^52 an integer; every value below is exact).
//   * m = floor(log2(X / Y)) with X = 2S + e and Y = 1.5 e.  For positive
//     normal binary64 values, bits(X) - bits(Y) = 2^52 (E_X - E_Y) + (F_X - F_Y),
//     so its floor quotient by 2^52 is E_X - E_Y, less one exactly when the
//     significand of X is below that of Y: floor(log2(X / Y)).  X and Y are
//     taken scaled by 2^-1000 (exact, still normal, biased exponents between
//     23 and 79): their patterns are then below 2^59, and shifted right by 27
//     they fit 32 bits.  Y = 3 e / 2 has at most 26 significant bits (e at
//     most 24), so its pattern is a multiple of 2^27 and
//         m = floor((floor(bits(X) / 2^27) - bits(Y) / 2^27) / 2^25),
//     two funnel shifts and a 32-bit difference.
//   * [2S < 3e] is e > tau, tau the largest binary32 value not above
//     floor(2S / 3): e is an integer held exactly in binary32.
// The empty asm hides the pattern's origin so that the compiler converts it
// to binary64 here rather than keeping the conversions of the I-Exp pass (two
// registers per key) alive across both passes.
constexpr double kCodeScale = 0x1p-1000;

struct RowState {
    double S2s;     // float path: 2S 2^-1000
    double sc;      // float path: 2^-1000, held in scalar registers (an fma
                    // cannot take it as a literal)
    float tau;      // float path: largest binary32 value <= floor(2S / 3)
    RowSum rs;      // integer path
};

// floor(bits(v) / 2^27) mod 2^32 of a binary64 value
__device__ __forceinline__ uint32_t bits_shr27(double v) {
    const uint64_t b = (uint64_t)__double_as_longlong(v);
    return __builtin_amdgcn_alignbit((uint32_t)(b >> 32), (uint32_t)b, 27);
}

// (floor(bits(X 2^-1000) / 2^27), bits(Y 2^-1000) / 2^27) of one key
__device__ __forceinline__ void code_bits(int ebits, const RowState& st, uint32_t& ax,
                                          uint32_t& ay, float& e) {
    asm volatile("" : "+v"(ebits));
    e = __int_as_float(ebits);
    const double ed = (double)e;
    ax = bits_shr27(fma(ed, st.sc, st.S2s));
    ay = bits_shr27(ed * (1.5 * kCodeScale));
}

__device__ __forceinline__ int code_f(int ebits, const RowState& st, int top) {
    uint32_t ax, ay;
    float e;
    code_bits(ebits, st, ax, ay, e);
    const int m = (int)((ax - ay) >> 25);
    return min(m, top) - (e > st.tau ? 1 : 0);
}

// top - code for top <= 15: with kr = (top + 1) 2^25 - 1, the saturated
// difference kr - (ax - ay) = (top - m) 2^25 + (2^25 - 1 - (ax - ay) mod 2^25)
// has max(top - m, 0) as its quotient by 2^25 (ay + kr stays below 2^32: the
// biased exponent of Y 2^-1000 is below 80).  min(m, top) - [2S < 3e] is
// top minus that quotient minus the comparison.
__device__ __forceinline__ uint32_t code_rev_f(int ebits, const RowState& st, uint32_t kr) {
    uint32_t ax, ay;
    float e;
    code_bits(ebits, st, ax, ay, e);
    const uint32_t r = __builtin_elementwise_sub_sat(ay + kr, ax) >> 25;
    return r + (e > st.tau ? 1u : 0u);
}

// Largest binary32 value <= floor(S2 / 3), S2 an integer below 2^53, with no
// division: q0 = floor(S2 RN(1/3)) is floor(S2 / 3) or one less (RN(1/3)
// is below 1/3 by at most 2^-55, so the product falls short of S2 / 3 by at
// most 1/4 before its rounding, itself at most 1/4 either way below 2^52),
// and the exact remainder S2 - 3 q0 (one fma; all values integers below
// 2^53) tells which.  The conversion to binary32 rounds to nearest and is
// stepped down when it lands above.
__device__ __forceinline__ float third_floor_f32(double S2) {
    double q = floor(S2 * (1.0 / 3.0));
    const double r = fma(-3.0, q, S2);
    q = r >= 3.0 ? q + 1.0 : q;
    const float f = (float)q;
    return (double)f > q ? __int_as_float(__float_as_int(f) - 1) : f;
}

// Wavefronts per SIMD the register allocation aims for: the logits of NC chunks
// take 8 NC registers per lane.
constexpr int lis_waves_per_simd(int NC) { return NC <= 8 ? 3 : (NC <= 12 ? 2 : 1); }

// ---------------------------------------------------------------------------
// Per-tile steps shared by the kernels.  lg holds the logits of a lane's
// keys; after tile_iexp it holds e (float path, as bits) or qL with z in zb
// (integer path); masked keys hold 0 there.  NT = elements of the last chunk
// that carry keys (4 with the half tail, else 8).
// ---------------------------------------------------------------------------

template <int NC>
__device__ __forceinline__ int tile_max(const int (&lg)[NC][8]) {
    int mx = INT_MIN;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
#pragma unroll
        for (int t = 0; t < 8; t += 2) mx = max(mx, max(lg[c][t], lg[c][t + 1]));
    }
    return row4_max(mx);
}

template <int NC, bool FP, int NT, bool P0 = false>
__device__ __forceinline__ RowState tile_iexp(int (&lg)[NC][8], uint32_t (&zb)[NC][2],
                                              const LisConsts& k) {
    const int mx = tile_max<NC>(lg);
    RowState st;
    if constexpr (FP) {
        // Four partial sums: every partial sum is an integer below 2^53, so the
        // binary64 additions are exact in any order (one serial chain would
        // make the scheduler hold every converted term in registers).
        double part[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
        for (int c = 0; c < NC; ++c) {
#pragma unroll
            for (int t = 0; t < (c < NC - 1 ? 8 : NT); ++t) {
                const int v = lg[c][t];
                float e = iexp_f<P0>(v, mx, k);
                if (c == NC - 1) e = v != INT_MIN ? e : 0.0f;
                part[t & 3] += (double)e;
                lg[c][t] = __float_as_int(e);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        double sum = (part[0] + part[1]) + (part[2] + part[3]);
        sum = row4_sum(sum);
        const double S2 = 2.0 * sum;
        st.S2s = S2 * kCodeScale;
        st.sc = kCodeScale;
        asm volatile("" : "+s"(st.sc));
        st.tau = third_floor_f32(S2);
    } else {
        uint64_t sum = 0;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            zb[c][0] = zb[c][1] = 0;
#pragma unroll
            for (int t = 0; t < (c < NC - 1 ? 8 : NT); ++t) {
                const int v = lg[c][t];
                const uint32_t u = min((uint32_t)mx - (uint32_t)v, k.u_max);
                const uint32_t z =
                    (uint32_t)(((uint64_t)((u << k.pre) & 0xFFFFFFu) * (uint64_t)k.magic) >> 32);
                const uint32_t w = __umul24(z, k.d_ln2) + (k.qb - u);
                const uint32_t qL = __umul24(w, w) + k.qc;
                const uint64_t e = (uint64_t)qL << (k.n - (int)z);
                if (c < NC - 1) {
                    sum += e;
                    lg[c][t] = (int)qL;
                } else {
                    const bool valid = v != INT_MIN;
                    sum += valid ? e : 0ull;
                    lg[c][t] = valid ? (int)qL : 0;
                }
                zb[c][t >> 2] |= z << (8 * (t & 3));
            }
        }
        st.rs = row_sum(sum, k);
    }
    return st;
}

// Codes of chunk c; in the last chunk masked keys (held as 0) get code 0 and
// the entries past NT are 0.
template <int NC, bool FP, int NT>
__device__ __forceinline__ void chunk_codes(int (&code)[8], const int (&lg)[NC][8],
                                            const uint32_t (&zb)[NC][2], const RowState& st,
                                            const LisConsts& k, int c) {
    const bool last = c == NC - 1;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
        if (last && t >= NT) {
            code[t] = 0;
            continue;
        }
        int cd;
        if constexpr (FP) {
            cd = code_f(lg[c][t], st, k.top);
        } else {
            const uint32_t z = (zb[c][t >> 2] >> (8 * (t & 3))) & 0xFFu;
            cd = lis_code((uint32_t)lg[c][t], z, st.rs, k);
        }
        code[t] = (last && lg[c][t] == 0) ? 0 : cd;
    }
}

// bf16 operand of P = 2^(N - code) for chunk c (masked keys 0), as four
// dwords holding the pairs (t, t + 1).  Float path: the bf16 pattern of
// 2^(N - code) is (127 + N - code) << 7, built from code_rev_f.
template <int NC, bool FP, int NT>
__device__ __forceinline__ u32x4 chunk_pbits(const int (&lg)[NC][8], const uint32_t (&zb)[NC][2],
                                             const RowState& st, const LisConsts& k, int c) {
    const bool last = c == NC - 1;
    if constexpr (FP) {
        const uint32_t kr = ((uint32_t)(k.top + 1) << 25) - 1u;
        uint32_t ex[8];
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            if (last && t >= NT) {
                ex[t] = 0;
                continue;
            }
            const uint32_t x = 127u + code_rev_f(lg[c][t], st, kr);
            ex[t] = (last && lg[c][t] == 0) ? 0u : x;
        }
        return u32x4{(ex[0] | (ex[1] << 16)) << 7, (ex[2] | (ex[3] << 16)) << 7,
                     (ex[4] | (ex[5] << 16)) << 7, (ex[6] | (ex[7] << 16)) << 7};
    } else {
        const float ptop = (float)(1 << k.top);
        float P[8];
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            if (last && t >= NT) {
                P[t] = 0.0f;
                continue;
            }
            const uint32_t z = (zb[c][t >> 2] >> (8 * (t & 3))) & 0xFFu;
            const int cd = lis_code((uint32_t)lg[c][t], z, st.rs, k);
            const float p = __builtin_ldexpf(ptop, -cd);
            P[t] = (last && lg[c][t] == 0) ? 0.0f : p;
        }
        return u32x4{bf16_pair(P[0], P[1]), bf16_pair(P[2], P[3]), bf16_pair(P[4], P[5]),
                     bf16_pair(P[6], P[7])};
    }
}

// acc[dt] += P x V^T for chunk c (cs: its index inside the current V^T stage).
// TR = false: acc[dt] is the 16 x 16 output block (rows i0.., columns 16 dt..)
// in the matrix cores' layout, lane (r, kg) holding rows 4 kg .. 4 kg + 3 of
// column 16 dt + r.  TR = true: the operands swap roles, so the instruction
// forms the transposed block V^T P^T from the same products and sums, and lane
// (r, kg) holds columns 16 dt + 4 kg .. + 3 of row i0 + r: four consecutive
// int32 of one output row, one 16-byte store.
template <int DTMAX, bool HALFMMA, bool TR = false>
__device__ __forceinline__ void chunk_mfma(f32x4 (&acc)[DTMAX], u32x4 pb, const uint16_t* vt,
                                           int ld, int cs, int r, int kg) {
    if constexpr (HALFMMA) {
        const i16x4 A = __builtin_bit_cast(i16x4, u32x2{pb.x, pb.y});
#pragma unroll
        for (int dt = 0; dt < DTMAX; ++dt) {
            const u32x2 bv = *reinterpret_cast<const u32x2*>(vt + (16 * dt + r) * ld + 32 * cs + 8 * kg);
            const i16x4 B = __builtin_bit_cast(i16x4, bv);
            if constexpr (TR)
                acc[dt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(B, A, acc[dt], 0, 0, 0);
            else
                acc[dt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(A, B, acc[dt], 0, 0, 0);
        }
    } else {
        const bf16x8 A = __builtin_bit_cast(bf16x8, pb);
#pragma unroll
        for (int dt = 0; dt < DTMAX; ++dt) {
            const u32x4 bv = *reinterpret_cast<const u32x4*>(vt + (16 * dt + r) * ld + 32 * cs + 8 * kg);
            const bf16x8 B = __builtin_bit_cast(bf16x8, bv);
            if constexpr (TR)
                acc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(B, A, acc[dt], 0, 0, 0);
            else
                acc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, B, acc[dt], 0, 0, 0);
        }
    }
}

// Output of transposed blocks (chunk_mfma with TR): lane (r, kg) writes
// out[g][i0 + r][16 dt + 4 kg + q] = acc[dt][q].  vec (d % 4 == 0, 16-byte
// aligned out): one 16-byte store per (row, dt), the four lanes of a row
// covering 64 contiguous bytes.  Streaming stores: the output is not read
// again here.
template <int DTMAX>
__device__ __forceinline__ void store_out_t(const f32x4 (&acc)[DTMAX], const LisArgs& a, int64_t g,
                                            int i0, int r, int kg, bool vec) {
    typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
    const int row = i0 + r;
    if (row >= a.Lq) return;
    int32_t* orow = a.out + (g * a.Lq + row) * (int64_t)a.d;
#pragma unroll
    for (int dt = 0; dt < DTMAX; ++dt) {
        const int col = 16 * dt + 4 * kg;
        if (col >= a.d) continue;
        if (vec) {
            const i32x4 v = {(int32_t)acc[dt][0], (int32_t)acc[dt][1], (int32_t)acc[dt][2],
                             (int32_t)acc[dt][3]};
            __builtin_nontemporal_store(v, reinterpret_cast<i32x4*>(orow + col));
        } else {
#pragma unroll
            for (int q = 0; q < 4; ++q)
                if (col + q < a.d) orow[col + q] = (int32_t)acc[dt][q];
        }
    }
}

// out[g][i0 + 4 kg + q][16 dt + r] = acc[dt][q]
template <int DTMAX>
__device__ __forceinline__ void store_out(const f32x4 (&acc)[DTMAX], const LisArgs& a, int64_t g,
                                          int i0, int r, int kg) {
#pragma unroll
    for (int dt = 0; dt < DTMAX; ++dt) {
        const int col = 16 * dt + r;
        if (col >= a.d) continue;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int orow = i0 + 4 * kg + q;
            if (orow < a.Lq) a.out[(g * a.Lq + orow) * (int64_t)a.d + col] = (int32_t)acc[dt][q];
        }
    }
}

// The same tile written through LDS: the wavefront's 16 x dpad block goes to
// its own LDS region ot (16 rows of 16 DTMAX + 4 dwords; the 4-dword pad makes
// the scattered writes conflict-free), then each store instruction writes
// whole output rows as 16-byte units, the tile being one contiguous range of
// out.  Needs d % 4 == 0 and a 16-byte aligned out.
template <int DTMAX>
constexpr int out_lds_dwords() { return 16 * (16 * DTMAX + 4); }

template <int DTMAX>
__device__ __forceinline__ void store_out_rows(const f32x4 (&acc)[DTMAX], int32_t* ot,
                                               const LisArgs& a, int64_t g, int i0, int lane,
                                               int r, int kg) {
    constexpr int LDO = 16 * DTMAX + 4;
    constexpr int UPR = 4 * DTMAX;    // 16-byte units per row
    typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
#pragma unroll
    for (int dt = 0; dt < DTMAX; ++dt) {
#pragma unroll
        for (int q = 0; q < 4; ++q) ot[(4 * kg + q) * LDO + 16 * dt + r] = (int32_t)acc[dt][q];
    }
    int32_t* otile = a.out + (g * a.Lq + i0) * (int64_t)a.d;
    if (i0 + 16 <= a.Lq && a.d == 16 * DTMAX) {
        // a whole tile: 16 consecutive rows of d columns, one contiguous range
#pragma unroll
        for (int j = 0; j < UPR / 4; ++j) {
            const int u = lane + 64 * j;
            const int row = u / UPR;
            const int c4 = u - row * UPR;
            // streaming stores: the output is not read again here, and
            // keeping it out of L2 leaves room for the logits (measured: the
            // fused head 3 % faster; non-temporal logit loads are much
            // slower, since the two 64-byte halves of a line are read by two
            // consecutive load instructions)
            __builtin_nontemporal_store(*reinterpret_cast<const i32x4*>(ot + row * LDO + 4 * c4),
                                        reinterpret_cast<i32x4*>(otile + 4 * u));
        }
        return;
    }
#pragma unroll
    for (int j = 0; j < UPR / 4; ++j) {
        const int u = lane + 64 * j;
        const int row = u / UPR;
        const int c4 = u - row * UPR;
        const i32x4 v = *reinterpret_cast<const i32x4*>(ot + row * LDO + 4 * c4);
        if (i0 + row < a.Lq && 4 * c4 < a.d)
            __builtin_nontemporal_store(v, reinterpret_cast<i32x4*>(otile + row * a.d + 4 * c4));
    }
}

// Row pointers of row i of unit g and whether its last chunk can be read with
// full vectors (32 NC elements from the row start lie inside the tensors).
struct RowPtrs {
    const int32_t* row;
    const int32_t* brow;
    bool tail_vec;
};

template <int NC>
__device__ __forceinline__ RowPtrs row_ptrs(const LisArgs& a, const LisLaunch& p, int64_t g, int i) {
    RowPtrs rp;
    const int64_t roff = (g * a.Lq + i) * (int64_t)a.Lk;
    rp.row = a.logits + roff;
    const int64_t boff = a.bias ? ((g % a.Hb) * a.Lq + i) * (int64_t)a.Lk : 0;
    rp.brow = a.bias ? a.bias + boff : nullptr;
    rp.tail_vec = roff + 32 * NC <= p.n_logits && (!rp.brow || boff + 32 * NC <= p.n_bias);
    return rp;
}

// Row pointers inside one unit from its base offsets (unit kernel): the unit's
// logit and bias planes are computed once, rows are offsets into them.
struct UnitBase {
    int64_t loff;   // offset of the unit's logits
    int64_t boff;   // offset of its head's bias plane (0 without bias)
};

template <int NC>
__device__ __forceinline__ RowPtrs unit_row(const LisArgs& a, const LisLaunch& p, const UnitBase& ub,
                                            int i) {
    RowPtrs rp;
    const int64_t roff = ub.loff + (int64_t)i * a.Lk;
    rp.row = a.logits + roff;
    const int64_t boff = ub.boff + (int64_t)i * a.Lk;
    rp.brow = a.bias ? a.bias + boff : nullptr;
    rp.tail_vec = roff + 32 * NC <= p.n_logits && (!rp.brow || boff + 32 * NC <= p.n_bias);
    return rp;
}

// Loads chunks [C0, C1) of a lane's keys.
template <int NC, bool HALF, int C0 = 0, int C1 = NC, bool DEFER = false>
__device__ __forceinline__ void tile_load(int (&lg)[NC][8], const RowPtrs& rp, int kg, int Lk) {
#pragma unroll
    for (int c = C0; c < C1; ++c) {
        if (c < NC - 1) load_full(lg[c], rp.row, rp.brow, c, kg);
        else load_chunk<HALF, DEFER>(lg[NC - 1], rp.row, rp.brow, NC - 1, kg, Lk, rp.tail_vec);
    }
}

// ---------------------------------------------------------------------------
// Unit kernel: one workgroup per attention unit, V^T staged once (single
// stage), each wavefront walks the unit's 16-row tiles w', w' + 4, ... and
// prefetches its next tile's logits while it computes the current one.  The
// wave with the extra tiles rotates with the unit so that the SIMDs of a CU
// share the remainder.  Float path only.  HALF: the last chunk holds at most
// 16 keys and is contracted by the 16x16x16 MFMA.
// ---------------------------------------------------------------------------
// Prefetch of the next tile: its first PF chunks are requested right after
// the I-Exp pass of the current tile, and chunk PF + c right after chunk c of
// the current tile has gone through its MFMA (its registers are free by then),
// so the next tile is in flight without holding two tiles in registers.
// Rows of five or more chunks also defer the masking of the last chunk's keys
// past Lk to the chunk's use (mask_last): applied at the load, it made the
// wavefront wait for the whole next tile right after requesting its last
// chunk, before the current tile's output was stored.  Measured on the ViT-B/16
// shapes (768 x 197 x 197, events over 96 launches, same box): deferred masking
// with PF = 2 (156 VGPRs) 43.8-45.3 us against 45.4-46.9 us before; PF = 0 or 1
// 44.5-45.3, PF = 3 45.6, PF = 4 48.1 (168 VGPRs, spills); requesting the last
// chunk first no better than PF = 0.  The small-unit kernels keep the masking
// at the load and PF = 0: deferred, they spill at their 80-register bound.
// Both are taken by the fused kernels (the codes-only kernels of seven chunks
// spill more with the deferred masking), PF = 2 where it fits the 168
// registers of three wavefronts per SIMD: all but the widest (seven full
// chunks and d > 32), which keeps PF = 0.
constexpr bool unit_defer(int NC, bool FUSED) { return FUSED && NC >= 5; }
constexpr int unit_prefetch(int NC, bool FUSED, int DTMAX, bool HALF) {
    return unit_defer(NC, FUSED) && !(NC == 7 && DTMAX == 4 && !HALF) ? 2 : 0;
}

template <int NC, bool HALF, bool DEFER = false>
__device__ __forceinline__ void load_one_chunk(int (&lg)[NC][8], const RowPtrs& rp, int c, int kg,
                                               int Lk) {
    if (c < NC - 1) load_full(lg[c], rp.row, rp.brow, c, kg);
    else load_chunk<HALF, DEFER>(lg[NC - 1], rp.row, rp.brow, NC - 1, kg, Lk, rp.tail_vec);
}

// Maximum and sum over all 64 lanes: the four rows of sixteen lanes by the
// lane swaps, then within each row by DPP rotations (every lane ends with the
// total).  The sum is exact for integers below 2^53, in any order.
__device__ __forceinline__ int wave_max(int v) {
    v = row4_max(v);
    v = max(v, __builtin_amdgcn_update_dpp(0, v, 0x128, 0xF, 0xF, false));   // row_ror:8
    v = max(v, __builtin_amdgcn_update_dpp(0, v, 0x124, 0xF, 0xF, false));   // row_ror:4
    v = max(v, __builtin_amdgcn_update_dpp(0, v, 0x122, 0xF, 0xF, false));   // row_ror:2
    return max(v, __builtin_amdgcn_update_dpp(0, v, 0x121, 0xF, 0xF, false)); // row_ror:1
}

__device__ __forceinline__ double wave_sum(double v) {
    v = row4_sum(v);
#pragma unroll
    for (int s = 3; s >= 0; --s) {
        const uint64_t b = (uint64_t)__double_as_longlong(v);
        int lo = (int)(uint32_t)b, hi = (int)(uint32_t)(b >> 32);
        switch (s) {
            case 3: lo = __builtin_amdgcn_update_dpp(0, lo, 0x128, 0xF, 0xF, false);
                    hi = __builtin_amdgcn_update_dpp(0, hi, 0x128, 0xF, 0xF, false); break;
            case 2: lo = __builtin_amdgcn_update_dpp(0, lo, 0x124, 0xF, 0xF, false);
                    hi = __builtin_amdgcn_update_dpp(0, hi, 0x124, 0xF, 0xF, false); break;
            case 1: lo = __builtin_amdgcn_update_dpp(0, lo, 0x122, 0xF, 0xF, false);
                    hi = __builtin_amdgcn_update_dpp(0, hi, 0x122, 0xF, 0xF, false); break;
            default: lo = __builtin_amdgcn_update_dpp(0, lo, 0x121, 0xF, 0xF, false);
                     hi = __builtin_amdgcn_update_dpp(0, hi, 0x121, 0xF, 0xF, false); break;
        }
        v += __longlong_as_double((int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo));
    }
    return v;
}

// A tile of one row (the last tile of units of 16 m + 1 rows, rows of at most
// two chunks), at the cost of one key per lane instead of a 16-row tile's
// eight per chunk: lane l takes key l (I-Exp, the wavefront's maximum and
// sum, its code by the float path's threshold form), the bf16 bits of
// 2^(N - code) go to LDS at the key's position in the matrix cores' order, and
// the lanes of row 0 read them back as the A operand of the usual P x V^T
// products (the other rows zero).  Same values as the 16-row tile: the row's
// maximum, its exact sum and each key's code do not depend on the lane layout.
template <int NC, int DTMAX>
__device__ __forceinline__ void unit_row1(const LisArgs& a, const LisLaunch& p, const LisConsts& k,
                                          const uint16_t* vt, int32_t* ot, const UnitBase& ub,
                                          int64_t g, int i0, int lane, int r, int kg) {
    static_assert(NC <= 2, "one key per lane");
    const int j = lane;
    const bool key = j < a.Lk && j < 32 * NC;
    const int64_t off = (int64_t)i0 * a.Lk + j;
    int v = INT_MIN;
    if (key) v = a.logits[ub.loff + off] + (a.bias ? a.bias[ub.boff + off] : 0);
    const int mx = wave_max(v);
    const float e = key ? iexp_f(v, mx, k) : 0.0f;
    const double S2 = 2.0 * wave_sum((double)e);
    RowState st;
    st.S2s = S2 * kCodeScale;
    st.sc = kCodeScale;
    asm volatile("" : "+s"(st.sc));
    st.tau = third_floor_f32(S2);
    const uint32_t kr = ((uint32_t)(k.top + 1) << 25) - 1u;
    const uint32_t x = key ? (127u + code_rev_f(__float_as_int(e), st, kr)) << 7 : 0u;
    uint16_t* pl = reinterpret_cast<uint16_t*>(ot);
    if (j < 32 * NC) pl[32 * (j >> 5) + chunk_pos(j & 31)] = (uint16_t)x;
    __builtin_amdgcn_wave_barrier();
    f32x4 acc[DTMAX];
#pragma unroll
    for (int dt = 0; dt < DTMAX; ++dt) acc[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        const u32x4 w = *reinterpret_cast<const u32x4*>(pl + 32 * c + 8 * kg);
        const u32x4 pb = r == 0 ? w : u32x4{0u, 0u, 0u, 0u};
        chunk_mfma<DTMAX, false>(acc, pb, vt, p.ld, c, r, kg);
    }
    __builtin_amdgcn_wave_barrier();
    if (p.out_vec) store_out_rows<DTMAX>(acc, ot, a, g, i0, lane, r, kg);
    else store_out<DTMAX>(acc, a, g, i0, r, kg);
}

template <int NC, bool FUSED, int DTMAX, bool HALF, int WPU>
__device__ __forceinline__ void unit_tile(int (&cur)[NC][8], int (&nxt)[NC][8], const LisArgs& a,
                                          const LisLaunch& p, const LisConsts& k, const uint16_t* vt,
                                          int32_t* ot, const UnitBase& ub, int64_t g, int tile,
                                          int ntl, int lane, int r, int kg, uint32_t valid) {
    constexpr int NT = HALF ? 4 : 8;
    constexpr int PF = unit_prefetch(NC, FUSED, DTMAX, HALF);
    constexpr bool DF = unit_defer(NC, FUSED);
    const int i0 = 16 * tile;
    // Always prefetch (a conditional load would keep the stale buffer live
    // across the loop); past the last tile the current rows, still in cache,
    // are read again.
    const int nt = tile + WPU < ntl ? tile + WPU : tile;
    const RowPtrs rn = unit_row<NC>(a, p, ub, min(16 * nt + r, a.Lq - 1));
    uint32_t zb[NC][2];
    if (DF) mask_last<NC, NT>(cur, valid);
    const RowState st = tile_iexp<NC, true, NT>(cur, zb, k);
    tile_load<NC, HALF, 0, PF, DF>(nxt, rn, kg, a.Lk);
    if constexpr (FUSED) {
        f32x4 acc[DTMAX];
#pragma unroll
        for (int dt = 0; dt < DTMAX; ++dt) acc[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            const u32x4 pb = chunk_pbits<NC, true, NT>(cur, zb, st, k, c);
            if (HALF && c == NC - 1)
                chunk_mfma<DTMAX, true>(acc, pb, vt, p.ld, c, r, kg);
            else
                chunk_mfma<DTMAX, false>(acc, pb, vt, p.ld, c, r, kg);
            if (PF + c < NC) load_one_chunk<NC, HALF, DF>(nxt, rn, PF + c, kg, a.Lk);
            // keep each chunk's V^T reads next to its MFMAs (hoisting them all
            // would take 4 DTMAX registers per chunk)
            __builtin_amdgcn_sched_barrier(0);
        }
        if (p.out_vec) store_out_rows<DTMAX>(acc, ot, a, g, i0, lane, r, kg);
        else store_out<DTMAX>(acc, a, g, i0, r, kg);
    } else if (p.codes_ldw != 0) {
        // Dense code rows: the tile's rows are one contiguous span of the codes
        // tensor.  They are gathered in LDS at the span's offset from a dword
        // boundary (mis), then written as whole aligned dwords, the partial
        // dwords at both ends byte by byte.
        const int i = i0 + r;
        const int nbr = k.top > 15 ? a.Lk : (a.Lk + 1) >> 1;
        const int rows = min(16, a.Lq - i0);
        uint8_t* cl = reinterpret_cast<uint8_t*>(ot);
        uint8_t* span = a.codes + (g * a.Lq + i0) * (int64_t)nbr;
        const int mis = (int)(reinterpret_cast<uintptr_t>(span) & 3);
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            int code[8];
            chunk_codes<NC, true, NT>(code, cur, zb, st, k, c);
            if (i < a.Lq) store_codes_row(cl + mis + r * nbr, a.Lk, k.top, c, kg, code);
            if (PF + c < NC) load_one_chunk<NC, HALF, DF>(nxt, rn, PF + c, kg, a.Lk);
            __builtin_amdgcn_sched_barrier(0);
        }
        __builtin_amdgcn_wave_barrier();
        uint8_t* gb = span - mis;
        const int end = mis + rows * nbr;
        for (int p0 = 4 * lane; p0 < end; p0 += 256) {
            if (p0 >= mis && p0 + 4 <= end) {
                *reinterpret_cast<uint32_t*>(gb + p0) = *reinterpret_cast<const uint32_t*>(cl + p0);
            } else {
#pragma unroll
                for (int t = 0; t < 4; ++t)
                    if (p0 + t >= mis && p0 + t < end) gb[p0 + t] = cl[p0 + t];
            }
        }
        __builtin_amdgcn_wave_barrier();
    } else {
        const int i = i0 + r;
        uint8_t* crow = a.codes + (g * a.Lq + min(i, a.Lq - 1)) * (int64_t)a.ld_codes;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            int code[8];
            chunk_codes<NC, true, NT>(code, cur, zb, st, k, c);
            if (i < a.Lq) store_codes_row(crow, a.Lk, k.top, c, kg, code);
            if (PF + c < NC) load_one_chunk<NC, HALF, DF>(nxt, rn, PF + c, kg, a.Lk);
            __builtin_amdgcn_sched_barrier(0);
        }
    }
}

// Minimum wavefronts per SIMD the register allocation is held to (the second
// argument of __launch_bounds__): three for four wavefronts per unit (168
// registers); for the small units that take one or two, six where the kernel
// fits 80 registers (codes-only rows of one chunk), so that as many units are
// in flight as the CU holds, five for fused rows of up to two chunks with
// d <= 32 (96 registers: with the one-row tile path they spilled at 80; on
// the Swin-S shapes five and six measured the same without it), and four
// otherwise (128 registers).
constexpr int unit_waves_per_simd(int NC, bool FUSED, int DTMAX, int WPU) {
    return WPU == 4 ? 3 : (FUSED && NC <= 2 && DTMAX <= 2 ? 5 : (!FUSED && NC <= 1) ? 6 : 4);
}

// WPU wavefronts per unit (4, or fewer for units of few tiles, so that each
// wavefront walks several; V^T staged by those 64 WPU threads).
template <int NC, bool FUSED, int DTMAX, bool HALF, int WPU = 4>
__global__ __launch_bounds__(64 * WPU, unit_waves_per_simd(NC, FUSED, DTMAX, WPU)) void lis_unit_kernel(
    LisArgs a, LisLaunch p) {
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    uint16_t* vt = reinterpret_cast<uint16_t*>(smem);
    const int64_t g = blockIdx.x;
    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const int r = lane & 15;
    const int kg = lane >> 4;

    LisConsts k = a.k;
    k.u_max &= 0xFFFFFFu;
    k.d_ln2 &= 0xFFFFFFu;
    k.magic &= 0xFFFFFFu;

    StageRegs sr;
    if constexpr (FUSED)
        stage_load<64 * WPU>(sr, a.v + g * (int64_t)a.Lk * a.d, a.Lk, a.d, DTMAX, 0, 32 * NC, p.vec_ok);

    UnitBase ub;
    ub.loff = g * a.Lq * (int64_t)a.Lk;
    ub.boff = a.bias ? (g % a.Hb) * a.Lq * (int64_t)a.Lk : 0;
    // Fused rows of at most two chunks: a last tile of one row (units of
    // 16 m + 1 rows) is left out of the tile loop and taken by unit_row1 after
    // it, where neither tile buffer is live.
    constexpr bool kRow1 = FUSED && NC <= 2;
    const int ntl = kRow1 && (a.Lq & 15) == 1 ? p.ntiles - 1 : p.ntiles;
    int bufA[NC][8], bufB[NC][8];
    int tile = (wave + (int)(g % WPU)) % WPU;
    if (tile < ntl)
        tile_load<NC, HALF, 0, NC, unit_defer(NC, FUSED)>(
            bufA, unit_row<NC>(a, p, ub, min(16 * tile + r, a.Lq - 1)), kg, a.Lk);
    const uint32_t valid = unit_defer(NC, FUSED) ? last_valid<NC>(kg, a.Lk) : 0xFFu;
    if constexpr (FUSED) {
        stage_store<64 * WPU>(sr, vt, p.ld, DTMAX, 32 * NC, a.zp_v);
        __syncthreads();
    }
    // LDS per wavefront: the output transpose (fused) or the tile's code rows
    int32_t* ot = FUSED ? reinterpret_cast<int32_t*>(smem + p.vt_bytes) + wave * out_lds_dwords<DTMAX>()
                        : reinterpret_cast<int32_t*>(smem + wave * p.codes_ldw);
    while (tile < ntl) {
        unit_tile<NC, FUSED, DTMAX, HALF, WPU>(bufA, bufB, a, p, k, vt, ot, ub, g, tile, ntl, lane, r,
                                               kg, valid);
        tile += WPU;
        if (tile >= ntl) break;
        unit_tile<NC, FUSED, DTMAX, HALF, WPU>(bufB, bufA, a, p, k, vt, ot, ub, g, tile, ntl, lane, r,
                                               kg, valid);
        tile += WPU;
    }
    if constexpr (kRow1) {
        if (tile == ntl && ntl < p.ntiles)
            unit_row1<NC, DTMAX>(a, p, k, vt, ot, ub, g, 16 * tile, lane, r, kg);
    }
}

// ---------------------------------------------------------------------------
// Tile kernel: a workgroup of four wavefronts owns one unit g and 64
// consecutive query rows.  FUSED = false: codes only.  FUSED = true: A x V by
// MFMA.  MULTI: V^T does not fit one LDS stage and is staged chunk range by
// chunk range.  FP: float path.  NC = number of 32-key chunks exactly
// (32 (NC - 1) < Lk <= 32 NC): every chunk but the last is full, so only the
// last one carries per-key masks.  DTMAX = 16-column output tiles, exactly
// dpad / 16.
// ---------------------------------------------------------------------------
template <int NC, bool FUSED, bool MULTI, int DTMAX, bool FP>
__global__ __launch_bounds__(kBlock, lis_waves_per_simd(NC)) void lis_kernel(LisArgs a,
                                                                            LisLaunch p) {
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    uint16_t* vt = reinterpret_cast<uint16_t*>(smem);
    const int64_t total = a.G * (int64_t)p.ntiles;
    const int64_t lb = xcd_remap(blockIdx.x, total);
    const int64_t g = lb / p.ntiles;
    const int tile = (int)(lb - g * p.ntiles);
    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const int r = lane & 15;
    const int kg = lane >> 4;
    const int i0 = tile * kRowsPerBlock + wave * 16;
    const int Lk = a.Lk;
    const bool active = i0 < a.Lq;

    LisConsts k = a.k;
    k.d_ln2 &= 0xFFFFFFu;
    k.magic &= 0xFFFFFFu;
    k.u_max &= 0xFFFFFFu;

    const int i = min(i0 + r, a.Lq - 1);
    const int8_t* vg = FUSED ? a.v + g * (int64_t)Lk * a.d : nullptr;

    StageRegs sr;
    if (FUSED) stage_load(sr, vg, Lk, a.d, p.ncg, 0, min(p.kb, NC * 32), p.vec_ok);

    int lg[NC][8];
    tile_load<NC, false>(lg, row_ptrs<NC>(a, p, g, i), kg, Lk);

    if (FUSED) stage_store(sr, vt, p.ld, p.ncg, min(p.kb, NC * 32), a.zp_v);

    uint32_t zb[NC][2];
    RowState st;
    if (active || MULTI) st = tile_iexp<NC, FP, 8>(lg, zb, k);
    if (FUSED) __syncthreads();   // V^T is visible
    if (!MULTI && !active) return;

    const bool row_ok = (i0 + r) < a.Lq;
    uint8_t* crow = FUSED ? nullptr : a.codes + (g * a.Lq + i) * (int64_t)a.ld_codes;
    f32x4 acc[DTMAX];
    if (FUSED) {
#pragma unroll
        for (int dt = 0; dt < DTMAX; ++dt) acc[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    const int cps = p.kb >> 5;  // chunks per V^T stage

#pragma unroll
    for (int c = 0; c < NC; ++c) {
        int cs = c;
        if (FUSED && MULTI) {
            const int stage = c / cps;
            cs = c - stage * cps;
            if (c > 0 && cs == 0) {
                __syncthreads();
                stage_vt(vt, p.ld, vg, Lk, a.d, p.ncg, stage * p.kb,
                         min(p.kb, NC * 32 - stage * p.kb), a.zp_v, p.vec_ok);
                __syncthreads();
            }
        }
        if (FUSED) {
            const u32x4 pb = chunk_pbits<NC, FP, 8>(lg, zb, st, k, c);
            chunk_mfma<DTMAX, false>(acc, pb, vt, p.ld, cs, r, kg);
            __builtin_amdgcn_sched_barrier(0);
        } else {
            int code[8];
            chunk_codes<NC, FP, 8>(code, lg, zb, st, k, c);
            if (row_ok) store_codes_row(crow, Lk, k.top, c, kg, code);
        }
    }

    if (FUSED && active) {
        int32_t* ot = reinterpret_cast<int32_t*>(smem + p.vt_bytes) + wave * out_lds_dwords<DTMAX>();
        if (p.out_vec) {
            store_out_rows<DTMAX>(acc, ot, a, g, i0, lane, r, kg);
        } else {
            store_out<DTMAX>(acc, a, g, i0, r, kg);
        }
    }
}

// Launch of the tile kernel for exactly NC chunks; the host has checked that
// dtm is 2 or 4 for fused calls (d <= 64).  MULTI follows from NC and dtm.
// Longest rows (in 32-key chunks) of the fused tile kernels.  Beyond 9 chunks
// the stream kernel, which re-reads the logits instead of holding them, is
// faster (d = 64, 64 square units, on one MI355X: 300 keys 30 against 36 us,
// 384 keys 41 against 61 us); up to 9 chunks the tile kernels are (288 keys
// 15 against 29 us, 240 keys 10 against 19 us).
constexpr int kRegsFusedMaxNC = 9;

template <int NC>
hipError_t launch_lis_nc(bool fused, int dtm, bool fp, const LisArgs& a, const LisLaunch& p,
                         dim3 grid, size_t lds, hipStream_t s) {
#define FQ_LIS(FUSED, MULTI, DTM, FP) \
    launch_kernel(lis_kernel<NC, FUSED, MULTI, DTM, FP>, grid, dim3(kBlock), lds, s, a, p)
    constexpr bool kMulti2 = NC * 32 > vt_stage_keys(32);
    constexpr bool kMulti4 = NC * 32 > vt_stage_keys(64);
    if (!fused) {
        if (fp) FQ_LIS(false, false, 1, true);
        else FQ_LIS(false, false, 1, false);
    } else if constexpr (NC > kRegsFusedMaxNC) {
        return hipErrorInvalidValue;    // longer fused rows take the stream kernel
    } else if (dtm == 2) {
        if (fp) FQ_LIS(true, kMulti2, 2, true);
        else FQ_LIS(true, kMulti2, 2, false);
    } else {
        if (fp) FQ_LIS(true, kMulti4, 4, true);
        else FQ_LIS(true, kMulti4, 4, false);
    }
#undef FQ_LIS
    return hipGetLastError();
}

// Launch of the unit kernel for exactly NC chunks (NC <= kUnitMaxNC).
constexpr int kUnitMaxNC = 7;

template <int NC, int WPU>
hipError_t launch_unit_nc_w(bool fused, int dtm, bool half, const LisArgs& a, const LisLaunch& p,
                            size_t lds, hipStream_t s) {
#define FQ_UNIT(FUSED, DTM, HALF)                                                                  \
    launch_kernel(lis_unit_kernel<NC, FUSED, DTM, HALF, WPU>, dim3((unsigned)a.G), dim3(64 * WPU), \
                  lds, s, a, p)
    if (!fused) {
        if (half) FQ_UNIT(false, 1, true);
        else FQ_UNIT(false, 1, false);
    } else if (dtm == 2) {
        if (half) FQ_UNIT(true, 2, true);
        else FQ_UNIT(true, 2, false);
    } else {
        if (half) FQ_UNIT(true, 4, true);
        else FQ_UNIT(true, 4, false);
    }
#undef FQ_UNIT
    return hipGetLastError();
}

// wpu: wavefronts per unit, 1 or 2 for rows of up to 4 chunks, else 4.
template <int NC>
hipError_t launch_unit_nc(bool fused, int dtm, bool half, int wpu, const LisArgs& a,
                          const LisLaunch& p, size_t lds, hipStream_t s) {
    if constexpr (NC <= 4) {
        if (wpu == 1) return launch_unit_nc_w<NC, 1>(fused, dtm, half, a, p, lds, s);
        if (wpu == 2) return launch_unit_nc_w<NC, 2>(fused, dtm, half, a, p, lds, s);
    }
    return launch_unit_nc_w<NC, 4>(fused, dtm, half, a, p, lds, s);
}

// Per chunk-count launchers, instantiated in lis_inst_lo.hip (1..10 chunks),
// lis_inst_hi.hip (11..20 chunks) and lis_inst_unit.hip (unit kernel, 1..7).
hipError_t launch_lis_regs_lo(int nc, bool fused, int dtm, bool fp, const LisArgs& a,
                              const LisLaunch& p, dim3 grid, size_t lds, hipStream_t stream);
hipError_t launch_lis_regs_hi(int nc, bool fused, int dtm, bool fp, const LisArgs& a,
                              const LisLaunch& p, dim3 grid, size_t lds, hipStream_t stream);
hipError_t launch_lis_unit(int nc, bool fused, int dtm, bool half, int wpu, const LisArgs& a,
                           const LisLaunch& p, size_t lds, hipStream_t stream);

}  // namespace lis
}  // namespace fqvit
