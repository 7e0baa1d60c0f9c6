// Device code of the Log-Int-Softmax attention kernels for gfx950 (Supplement A.2: Algorithm 1 I-Exp,
// Algorithm 2 I-Log2 and Log-Int-Softmax, the clip of the LIS equation; the
// BitShift product with V of Sec. 3.3 and its zero-point form).
//
// Work decomposition.  A workgroup of four wavefronts owns one attention unit
// g (image x window x head) and 64 consecutive query rows; each wavefront owns
// 16 rows.  Inside a wavefront, lane (r, kg) = (lane % 16, lane / 16) holds
// row r and, in every 32-key chunk c, the eight keys
//     32c + 4kg + t       (t = 0..3)   and   32c + 16 + 4kg + t   (t = 0..3),
// so each 16-byte load of a lane is contiguous and the four lanes of a row
// cover 64 contiguous bytes per load instruction.  The same eight keys are the
// eight k-slots the lane feeds to the 16x16x32 bf16 MFMA; V^T is staged in LDS
// with its keys permuted the same way, so the contraction pairs every key of
// the attention row with its own V row.
//
// Per row: max (lane-local, then two cross-lane shuffles), i-exp and the
// 64-bit sum, then the 4-bit code of every key.  The codes never leave the
// chip in the fused kernel: each becomes P = 2^(N - code) as a bf16 bit
// pattern and the chunk is multiplied with V^T by MFMA.  That product is
// exact: P and V - zp_V are exact in bf16, every product is an integer and
// every partial sum is an integer of magnitude below 2^24 (the codes of a row
// satisfy sum_j 2^-code_j < 1.5 + (Lk - 1)/2^15, so |out| <
// 255 * (1.5 * 2^15 + Lk) < 2^24 for Lk <= 4096), so fp32 accumulation in any
// order rounds nothing.
//
// The code needs no division.  With e = qL << s (qL = (q_p + q_b)^2 + q_c,
// s = n - z), the paper's r = round(S / e) (ties up) and I-Log2 satisfy
//     I-Log2(r) >= k   <=>   r >= T_k   <=>   2S + e >= 2 T_k e,
// T_1 = 2, T_k = 3 * 2^(k-2).  Writing Sp = floor(2S / 2^s), W = Sp + qL and
// Q = 3 qL this is Sp >= Q for k = 1 and W >= Q * 2^(k-1) for k >= 2, so the
// code is j + 1 - [Sp < Q] with j = floor(log2(W / Q)).  Because msb(W) is
// msb(2S) - s or one more, j is j0 - 1, j0 or j0 + 1 with
// j0 = msb(2S) - s - msb(Q) (msb(2S) once per row), and two exact 64-bit
// comparisons of W against Q 2^j0 and Q 2^(j0+1) settle it.
#pragma once

#include "fqvit_internal.h"

namespace fqvit {
namespace lis {

constexpr int kBlock = 256;        // four wavefronts
constexpr int kRowsPerBlock = 64;  // 16 rows per wavefront

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int32_t i32x4a4 __attribute__((ext_vector_type(4), aligned(4)));

// Block index -> logical tile so that the tiles of one unit run on one XCD
// (blocks are dealt round-robin to the eight XCDs) and share its L2.
__device__ __forceinline__ int64_t xcd_remap(int64_t b, int64_t total) {
    const int64_t per = total >> 3;
    if (b >= (per << 3)) return b;
    return (b & 7) * per + (b >> 3);
}

// floor(u / d) for u <= n d, with magic = floor(2^32 / (d << pre)) + 1 and
// n (d << pre)^2 < 2^32, (d << pre) > 256 (checked on the host): the 24-bit
// high multiply is exact under those bounds.
__device__ __forceinline__ uint32_t div_ln2(uint32_t u, const LisConsts& k) {
    const uint64_t prod = (uint64_t)((u << k.pre) & 0xFFFFFFu) * (uint64_t)(k.magic & 0xFFFFFFu);
    return (uint32_t)(prod >> 32);
}

__device__ __forceinline__ uint16_t bf16_of_int(int x) {
    // exact for |x| <= 256
    return (uint16_t)(__float_as_uint((float)x) >> 16);
}

// Position of key j (0..31) of a chunk in the permuted order: the eight keys
// of lane group kg are contiguous.
__device__ __forceinline__ int chunk_pos(int j) {
    return ((j & 15) >> 2) * 8 + ((j >> 4) << 2) + (j & 3);
}

// Staging of keys [k0, k0 + kcnt) of V[g] into vt[dd][pos] as bf16 bits of
// v - zp (kcnt a multiple of 32, dpad a multiple of 16).  A work item is a
// key pair and a group of 16 columns: two 16-byte loads (V rows jj and jj + 1)
// and sixteen 32-bit LDS stores of bf16 pairs.  The key pair runs fastest
// across the threads, so the stores of a wavefront hit consecutive dwords
// (bank-conflict free).  All loads of a thread are issued before its stores.
// A stage holds at most 40 KB: kcnt * dpad / 32 <= 640 items, at most
// kStageItems per thread of a 256-thread workgroup.
constexpr int kStageItems = 3;

struct StageRegs {
    u32x4 w0[kStageItems], w1[kStageItems];
};

__device__ __forceinline__ u32x4 load_v16(const int8_t* vrow, int dd, int d, bool vec_ok) {
    if (vec_ok) return *reinterpret_cast<const u32x4*>(vrow + dd);
    u32x4 w = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int q = 0; q < 16; ++q)
        if (dd + q < d) w[q >> 2] |= (uint32_t)(uint8_t)vrow[dd + q] << (8 * (q & 3));
    return w;
}

__device__ __forceinline__ void stage_load(StageRegs& sr, const int8_t* vg, int Lk, int d,
                                           int ncg, int k0, int kcnt, bool vec_ok) {
    const int npairs = kcnt >> 1;
    const int nitems = npairs * ncg;
#pragma unroll
    for (int it = 0; it < kStageItems; ++it) {
        const int idx = (int)threadIdx.x + it * (int)blockDim.x;
        const int cg = idx / npairs;
        const int j = k0 + 2 * (idx - cg * npairs);
        const int dd = 16 * cg;
        const bool ok = idx < nitems && dd < d;
        sr.w0[it] = (ok && j < Lk) ? load_v16(vg + (int64_t)j * d, dd, d, vec_ok) : u32x4{0u, 0u, 0u, 0u};
        sr.w1[it] = (ok && j + 1 < Lk) ? load_v16(vg + (int64_t)(j + 1) * d, dd, d, vec_ok)
                                       : u32x4{0u, 0u, 0u, 0u};
    }
}

__device__ __forceinline__ void stage_store(const StageRegs& sr, uint16_t* vt, int ld, int ncg,
                                            int kcnt, int zp) {
    const int npairs = kcnt >> 1;
    const int nitems = npairs * ncg;
#pragma unroll
    for (int it = 0; it < kStageItems; ++it) {
        const int idx = (int)threadIdx.x + it * (int)blockDim.x;
        if (idx >= nitems) continue;
        const int cg = idx / npairs;
        const int jj = 2 * (idx - cg * npairs);
        const int p0 = (jj & ~31) + chunk_pos(jj & 31);   // jj even: p0 + 1 is key jj + 1
#pragma unroll
        for (int q = 0; q < 16; ++q) {
            // Keys past Lk and columns past d hold -zp: the keys get P = 0 and
            // the columns are never stored, so any finite value is harmless.
            const int x0 = (int)(int8_t)(sr.w0[it][q >> 2] >> (8 * (q & 3)));
            const int x1 = (int)(int8_t)(sr.w1[it][q >> 2] >> (8 * (q & 3)));
            *reinterpret_cast<uint32_t*>(vt + (16 * cg + q) * ld + p0) =
                (uint32_t)bf16_of_int(x0 - zp) | ((uint32_t)bf16_of_int(x1 - zp) << 16);
        }
    }
}

// Staging of one V^T stage by the whole workgroup (used between stages).
__device__ __forceinline__ void stage_vt(uint16_t* vt, int ld, const int8_t* vg, int Lk, int d,
                                         int ncg, int k0, int kcnt, int zp, bool vec_ok) {
    StageRegs sr;
    stage_load(sr, vg, Lk, d, ncg, k0, kcnt, vec_ok);
    stage_store(sr, vt, ld, ncg, kcnt, zp);
}

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
// vectors and masked afterwards.
__device__ __forceinline__ void load_chunk(int (&dst)[8], const int32_t* row, const int32_t* brow,
                                           int c, int kg, int Lk, bool vec_ok) {
    const int k0 = 32 * c + 4 * kg;
    const int k1 = k0 + 16;
    if (vec_ok || k1 + 4 <= Lk) {
        load_full(dst, row, brow, c, kg);
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            const int key = (t < 4 ? k0 : k1 - 4) + t;
            if (key >= Lk) dst[t] = INT_MIN;
        }
    } else {
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            const int key = (t < 4 ? k0 : k1 - 4) + t;
            dst[t] = key < Lk ? row[key] + (brow ? brow[key] : 0) : INT_MIN;
        }
    }
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


// Keys of V^T per LDS stage for a padded head dimension dpad: at most 40 KB of
// LDS per workgroup so that several workgroups share a CU.
constexpr int vt_stage_keys(int dpad) { return (40960 / (2 * dpad) - 8) / 32 * 32; }

struct LisLaunch {
    int ntiles;     // row tiles of 64 per unit
    int kb;         // keys per V^T stage (multiple of 32)
    int ld;         // LDS row stride of V^T in bf16 elements
    int dpad;       // 16 * (power of two >= ceil(d / 16))
    int ncg;        // dpad / 16: 16-column groups of V
    int vec_ok;     // V rows read as 16-byte vectors (d % 16 == 0, 16-byte aligned V)
    int vt_bytes;   // LDS bytes of one V^T stage (0 for codes only)
    int64_t n_logits;  // elements of the logits tensor (G Lq Lk)
    int64_t n_bias;    // elements of the bias tensor (Hb Lq Lk), 0 without bias
};

// Per-row state after the I-Exp pass.
struct RowSum {
    uint64_t S2;    // 2 * sum_j e_j
    int rc;         // msb(S2) - 31 - n: j0 = rc + z + clz(3 qL)
};

__device__ __forceinline__ RowSum row_sum(uint64_t sum, const LisConsts& k) {
    sum += __shfl_xor(sum, 16, 64);
    sum += __shfl_xor(sum, 32, 64);
    RowSum rs;
    rs.S2 = sum << 1;
    rs.rc = (63 - __clzll((long long)rs.S2)) - 31 - k.n;
    return rs;
}

// I-Exp of one key (Algorithm 1): returns qL = (q_p + q_b)^2 + q_c and z; the
// i-exp value is e = qL << (n - z).
__device__ __forceinline__ uint32_t iexp_qL(int v, int mx, const LisConsts& k, uint32_t& z) {
    const uint32_t u = min((uint32_t)mx - (uint32_t)v, k.u_max);               // q <- max(q, n q_ln2)
    z = (uint32_t)(((uint64_t)((u << k.pre) & 0xFFFFFFu) * (uint64_t)k.magic) >> 32);  // floor(q / q_ln2)
    const uint32_t w = (k.qb - u + __umul24(z, k.d_ln2)) & 0xFFFFu;            // q_p + q_b
    return __umul24(w, w) + k.qc;
}

// bf16 exponent field (<< 7) of P = 2^(N - Attn_Q) for one key, from its qL,
// z and the row state.  Attn_Q = min(I-Log2(round(S / e)), N) via
// j = floor(log2(W / Q)) with W = floor(2S / 2^s) + qL, Q = 3 qL, s = n - z:
// msb(W) is msb(2S) - s or one more, so j is j0 - 1, j0 or j0 + 1 with
// j0 = msb(2S) - s - msb(Q), settled by two exact comparisons.
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

// Wavefronts per SIMD the register allocation aims for: the logits of NC chunks
// take 8 NC registers per lane.
constexpr int lis_waves_per_simd(int NC) { return NC <= 8 ? 3 : (NC <= 12 ? 2 : 1); }

// FUSED = false: codes only.  FUSED = true: A x V by MFMA.  MULTI: V^T does
// not fit one LDS stage.  PRE0: the I-Exp division needs no pre-shift.
// NC = number of 32-key chunks exactly (32 (NC - 1) < Lk <= 32 NC): every
// chunk but the last is full, so only the last one carries per-key masks.
// DTMAX = 16-column output tiles, exactly dpad / 16.
template <int NC, bool FUSED, bool MULTI, int DTMAX, bool PRE0>
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
    const int64_t roff = (g * a.Lq + i) * (int64_t)Lk;
    const int32_t* row = a.logits + roff;
    const int64_t boff = a.bias ? ((g % a.Hb) * a.Lq + i) * (int64_t)Lk : 0;
    const int32_t* brow = a.bias ? a.bias + boff : nullptr;
    const int8_t* vg = FUSED ? a.v + g * (int64_t)Lk * a.d : nullptr;
    const bool tail_vec = roff + 32 * NC <= p.n_logits && (!brow || boff + 32 * NC <= p.n_bias);

    StageRegs sr;
    if (FUSED) stage_load(sr, vg, Lk, a.d, p.ncg, 0, min(p.kb, NC * 32), p.vec_ok);

    int lg[NC][8];
#pragma unroll
    for (int c = 0; c < NC - 1; ++c) load_full(lg[c], row, brow, c, kg);
    load_chunk(lg[NC - 1], row, brow, NC - 1, kg, Lk, tail_vec);

    if (FUSED) stage_store(sr, vt, p.ld, p.ncg, min(p.kb, NC * 32), a.zp_v);

    uint32_t zb[NC][2];
    RowSum rs;
    if (active || MULTI) {
        // row maximum (masked keys hold INT_MIN)
        int mx = INT_MIN;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
#pragma unroll
            for (int t = 0; t < 8; t += 2) mx = max(mx, max(lg[c][t], lg[c][t + 1]));
        }
        mx = max(mx, __shfl_xor(mx, 16, 64));
        mx = max(mx, __shfl_xor(mx, 32, 64));

        // I-Exp (Algorithm 1): lg <- qL (0 for masked keys), zb <- z bytes; row sum of e.
        uint64_t sum = 0;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            zb[c][0] = zb[c][1] = 0;
#pragma unroll
            for (int t = 0; t < 8; ++t) {
                const int v = lg[c][t];
                const uint32_t u = min((uint32_t)mx - (uint32_t)v, k.u_max);
                const uint32_t up = PRE0 ? u : ((u << k.pre) & 0xFFFFFFu);
                const uint32_t z = (uint32_t)(((uint64_t)up * (uint64_t)k.magic) >> 32);
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
        rs = row_sum(sum, k);
    }
    if (FUSED) __syncthreads();   // V^T is visible
    if (!MULTI && !active) return;

    const int nbytes = (Lk + 1) >> 1;
    const bool row_ok = (i0 + r) < a.Lq;
    uint8_t* crow = FUSED ? nullptr : a.codes + (g * a.Lq + i) * (int64_t)a.ld_codes;
    f32x4 acc[DTMAX];
    if (FUSED) {
#pragma unroll
        for (int dt = 0; dt < DTMAX; ++dt) acc[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    const uint32_t ptop = (uint32_t)((127 + k.top) << 7);
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
        int code[8];
        uint32_t pbits[8];
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            const uint32_t qL = (uint32_t)lg[c][t];
            const uint32_t z = (zb[c][t >> 2] >> (8 * (t & 3))) & 0xFFu;
            const int cd = lis_code(qL, z, rs, k);
            const uint32_t pb = ptop - ((uint32_t)cd << 7);
            if (c < NC - 1) {
                code[t] = cd;
                pbits[t] = pb;
            } else {
                const bool valid = qL != 0;
                code[t] = valid ? cd : 0;
                pbits[t] = valid ? pb : 0u;
            }
        }
        if (!FUSED && row_ok) store_codes(crow, nbytes, c, kg, code);
        if (FUSED) {
            u32x4 av;
            av.x = pbits[0] | (pbits[1] << 16);
            av.y = pbits[2] | (pbits[3] << 16);
            av.z = pbits[4] | (pbits[5] << 16);
            av.w = pbits[6] | (pbits[7] << 16);
            const bf16x8 A = __builtin_bit_cast(bf16x8, av);
#pragma unroll
            for (int dt = 0; dt < DTMAX; ++dt) {
                const u32x4 bv = *reinterpret_cast<const u32x4*>(
                    vt + (16 * dt + r) * p.ld + 32 * cs + 8 * kg);
                acc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, __builtin_bit_cast(bf16x8, bv),
                                                                  acc[dt], 0, 0, 0);
            }
        }
    }

    if (FUSED && active) {
        // acc[dt][q] = out[row i0 + 4 kg + q][col 16 dt + r]
#pragma unroll
        for (int dt = 0; dt < DTMAX; ++dt) {
            const int col = 16 * dt + r;
            if (col >= a.d) continue;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int orow = i0 + 4 * kg + q;
                if (orow < a.Lq)
                    a.out[(g * a.Lq + orow) * (int64_t)a.d + col] = (int32_t)acc[dt][q];
            }
        }
    }
}

// Launch of the register kernel for exactly NC chunks; the host has checked
// that dtm is 2 or 4 for fused calls (d <= 64) and set multi when V^T needs
// more than one LDS stage.
template <int NC>
hipError_t launch_lis_nc(bool fused, bool multi, int dtm, bool pre0, const LisArgs& a,
                         const LisLaunch& p, dim3 grid, size_t lds, hipStream_t s) {
#define FQ_LIS(FUSED, MULTI, DTM, PRE0) \
    hipLaunchKernelGGL((lis_kernel<NC, FUSED, MULTI, DTM, PRE0>), grid, dim3(kBlock), lds, s, a, p)
    constexpr bool kMulti2 = NC * 32 > vt_stage_keys(32);
    constexpr bool kMulti4 = NC * 32 > vt_stage_keys(64);
    if (!fused) {
        FQ_LIS(false, false, 1, false);
    } else if (dtm == 2) {
        if (pre0) FQ_LIS(true, kMulti2, 2, true);
        else FQ_LIS(true, kMulti2, 2, false);
    } else {
        if (pre0) FQ_LIS(true, kMulti4, 4, true);
        else FQ_LIS(true, kMulti4, 4, false);
    }
#undef FQ_LIS
    (void)multi;
    return hipGetLastError();
}

// Register-kernel launchers, instantiated per chunk count in lis_inst_lo.hip
// (1..10 chunks) and lis_inst_hi.hip (11..20 chunks).
hipError_t launch_lis_regs_lo(int nc, bool fused, bool multi, int dtm, bool pre0,
                              const LisArgs& a, const LisLaunch& p, dim3 grid, size_t lds,
                              hipStream_t stream);
hipError_t launch_lis_regs_hi(int nc, bool fused, bool multi, int dtm, bool pre0,
                              const LisArgs& a, const LisLaunch& p, dim3 grid, size_t lds,
                              hipStream_t stream);

}  // namespace lis
}  // namespace fqvit
