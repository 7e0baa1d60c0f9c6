// Log-Int-Softmax attention for gfx950 (Supplement A.2: Algorithm 1 I-Exp,
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
// T_1 = 2, T_k = 3 * 2^(k-2).  Writing W = floor(2S / 2^s) + qL and Q = 3 qL
// this is W >= 4 qL for k = 1 and W >= Q * 2^(k-1) for k >= 2, so the code is
// floor(log2(W / Q)) + 1 when that is >= 2 and [W >= 4 qL] otherwise, where
// floor(log2(W / Q)) is msb(W) - msb(Q) minus one exact 64-bit comparison.
#include "fqvit_internal.h"

namespace fqvit {
namespace {

constexpr int kBlock = 256;        // four wavefronts
constexpr int kRowsPerBlock = 64;  // 16 rows per wavefront
constexpr uint32_t kMasked = 0xFFFFFFFFu;

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

// I-Exp of t = -u (u = max - v >= 0), Algorithm 1.  Returns the packed pair
// (w = q_p + q_b, z) and adds e = qL << (n - z) to sum.
__device__ __forceinline__ uint32_t iexp_pack(int v, int mx, const LisConsts& k, uint64_t& sum) {
    const uint32_t u = min((uint32_t)mx - (uint32_t)v, k.u_max);  // q <- max(q, n q_ln2)
    const uint32_t z = div_ln2(u, k);                             // z = floor(q / q_ln2)
    const uint32_t w = k.qb - u + z * k.d_ln2;                    // q_p + q_b
    const uint32_t qL = w * w + k.qc;                             // (q_p + q_b)^2 + q_c
    sum += (uint64_t)qL << (k.n - (int)z);                        // q_L << (n - z)
    return w | (z << 16);
}

// Attn_Q of one key from its packed (w, z) and S2 = 2 * sum.
__device__ __forceinline__ int lis_code(uint32_t pk, uint64_t S2, const LisConsts& k) {
    const uint32_t w = pk & 0xFFFFu;
    const int z = (int)(pk >> 16);
    const uint32_t qL = w * w + k.qc;
    const uint64_t W = (S2 >> (k.n - z)) + qL;
    const uint32_t Q = 3u * qL;
    int j = (63 - __clzll((long long)W)) - (31 - __clz((int)Q));
    j -= (W < ((uint64_t)Q << j)) ? 1 : 0;
    const int code = (j >= 1) ? (j + 1) : (W >= 4ull * qL ? 1 : 0);
    return min(code, k.top);
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

// Stage keys [k0, k0 + kcnt) of V[g] into vt[dd][pos] as bf16 bits of v - zp.
__device__ void stage_vt(uint16_t* vt, int ld, const int8_t* vg, int Lk, int d, int dpad,
                         int k0, int kcnt, int zp, bool dword_ok) {
    if (dword_ok) {
        // two keys x four columns per item: two dword loads, four 32-bit LDS stores
        const int ncol4 = dpad >> 2;
        const int nitems = (kcnt >> 1) * ncol4;
        for (int idx = threadIdx.x; idx < nitems; idx += blockDim.x) {
            const int jp = idx / ncol4;
            const int cq = idx - jp * ncol4;
            const int jj = 2 * jp;
            const int j = k0 + jj;
            const int dd = 4 * cq;
            uint32_t w0 = 0, w1 = 0;
            const bool col_ok = dd < d;
            if (col_ok && j < Lk) w0 = *reinterpret_cast<const uint32_t*>(vg + (int64_t)j * d + dd);
            if (col_ok && j + 1 < Lk) w1 = *reinterpret_cast<const uint32_t*>(vg + (int64_t)(j + 1) * d + dd);
            const int p0 = (jj & ~31) + chunk_pos(jj & 31);
            const int p1 = (jj & ~31) + chunk_pos((jj + 1) & 31);
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int a = (col_ok && j < Lk) ? (int)(int8_t)(w0 >> (8 * q)) - zp : 0;
                const int b = (col_ok && j + 1 < Lk) ? (int)(int8_t)(w1 >> (8 * q)) - zp : 0;
                vt[(dd + q) * ld + p0] = bf16_of_int(a);
                vt[(dd + q) * ld + p1] = bf16_of_int(b);
            }
        }
    } else {
        const int nitems = kcnt * dpad;
        for (int idx = threadIdx.x; idx < nitems; idx += blockDim.x) {
            const int jj = idx / dpad;
            const int dd = idx - jj * dpad;
            const int j = k0 + jj;
            const int x = (j < Lk && dd < d) ? (int)vg[(int64_t)j * d + dd] - zp : 0;
            vt[dd * ld + (jj & ~31) + chunk_pos(jj & 31)] = bf16_of_int(x);
        }
    }
}

// Load the 8 logits (+ bias) of lane (r, kg) in chunk c; masked keys get INT_MIN.
__device__ __forceinline__ void load_chunk(int (&dst)[8], const int32_t* row, const int32_t* brow,
                                           int c, int kg, int Lk) {
    const int k0 = 32 * c + 4 * kg;
    const int k1 = k0 + 16;
    if (k1 + 4 <= Lk) {
        const i32x4a4 a = *reinterpret_cast<const i32x4a4*>(row + k0);
        const i32x4a4 b = *reinterpret_cast<const i32x4a4*>(row + k1);
        dst[0] = a.x; dst[1] = a.y; dst[2] = a.z; dst[3] = a.w;
        dst[4] = b.x; dst[5] = b.y; dst[6] = b.z; dst[7] = b.w;
        if (brow) {
            const i32x4a4 ba = *reinterpret_cast<const i32x4a4*>(brow + k0);
            const i32x4a4 bb = *reinterpret_cast<const i32x4a4*>(brow + k1);
            dst[0] += ba.x; dst[1] += ba.y; dst[2] += ba.z; dst[3] += ba.w;
            dst[4] += bb.x; dst[5] += bb.y; dst[6] += bb.z; dst[7] += bb.w;
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

struct LisLaunch {
    int ntiles;     // row tiles of 64 per unit
    int kb;         // keys per V^T stage (multiple of 32)
    int ld;         // LDS row stride of V^T in bf16 elements
    int dpad;       // 16 * ceil(d / 16)
    int dword_ok;   // V rows dword aligned
};

// FUSED = false: codes only.  FUSED = true: A x V by MFMA, codes optional.
// NC = chunks held in registers (Lk <= 32 NC); DTMAX = 16-column tiles of the
// output held in accumulators (d <= 16 DTMAX).
template <int NC, bool FUSED, int DTMAX>
__global__ __launch_bounds__(kBlock) void lis_kernel(LisArgs a, LisLaunch p) {
    extern __shared__ uint16_t vt[];
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
    const int nc = (Lk + 31) >> 5;
    const int nstage = FUSED ? (nc * 32 + p.kb - 1) / p.kb : 0;
    const bool active = i0 < a.Lq;
    if (!FUSED && !active) return;

    const int i = min(i0 + r, a.Lq - 1);
    const int32_t* row = a.logits + (g * a.Lq + i) * (int64_t)Lk;
    const int32_t* brow = a.bias ? a.bias + ((g % a.Hb) * a.Lq + i) * (int64_t)Lk : nullptr;
    const int8_t* vg = FUSED ? a.v + g * (int64_t)Lk * a.d : nullptr;

    int lg[NC][8];
#pragma unroll
    for (int c = 0; c < NC; ++c)
        if (c < nc) load_chunk(lg[c], row, brow, c, kg, Lk);

    if (FUSED) {
        stage_vt(vt, p.ld, vg, Lk, a.d, p.dpad, 0, min(p.kb, nc * 32), a.zp_v, p.dword_ok);
        __syncthreads();
        if (nstage == 1 && !active) return;
    }

    // row maximum
    int mx = INT_MIN;
#pragma unroll
    for (int c = 0; c < NC; ++c)
        if (c < nc) {
#pragma unroll
            for (int t = 0; t < 8; ++t) mx = max(mx, lg[c][t]);
        }
    mx = max(mx, __shfl_xor(mx, 16, 64));
    mx = max(mx, __shfl_xor(mx, 32, 64));

    // I-Exp and the row sum
    const LisConsts k = a.k;
    uint64_t sum = 0;
#pragma unroll
    for (int c = 0; c < NC; ++c)
        if (c < nc) {
#pragma unroll
            for (int t = 0; t < 8; ++t) {
                const int v = lg[c][t];
                uint64_t s1 = 0;
                const uint32_t pk = iexp_pack(v, mx, k, s1);
                const bool valid = v != INT_MIN;
                sum += valid ? s1 : 0;
                lg[c][t] = valid ? (int)pk : (int)kMasked;
            }
        }
    sum += __shfl_xor(sum, 16, 64);
    sum += __shfl_xor(sum, 32, 64);
    const uint64_t S2 = sum << 1;

    const int nbytes = (Lk + 1) >> 1;
    const bool row_ok = (i0 + r) < a.Lq;
    uint8_t* crow = a.codes ? a.codes + (g * a.Lq + i) * (int64_t)a.ld_codes : nullptr;

    const int DT = p.dpad >> 4;
    f32x4 acc[DTMAX];
    if (FUSED) {
#pragma unroll
        for (int dt = 0; dt < DTMAX; ++dt) acc[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    int stage = 0;
    const int cps = p.kb >> 5;  // chunks per stage
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        if (c >= nc) break;
        if (FUSED && c > 0 && c % cps == 0) {
            ++stage;
            __syncthreads();
            stage_vt(vt, p.ld, vg, Lk, a.d, p.dpad, stage * p.kb, min(p.kb, nc * 32 - stage * p.kb),
                     a.zp_v, p.dword_ok);
            __syncthreads();
        }
        int code[8];
        uint32_t pbits[8];
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            const uint32_t pk = (uint32_t)lg[c][t];
            const bool valid = pk != kMasked;
            const int cd = lis_code(valid ? pk : 0u, S2, k);
            code[t] = valid ? cd : 0;
            pbits[t] = valid ? (uint32_t)(127 + k.top - cd) << 7 : 0u;
        }
        if (crow && row_ok) store_codes(crow, nbytes, c, kg, code);
        if (FUSED) {
            u32x4 av;
            av.x = pbits[0] | (pbits[1] << 16);
            av.y = pbits[2] | (pbits[3] << 16);
            av.z = pbits[4] | (pbits[5] << 16);
            av.w = pbits[6] | (pbits[7] << 16);
            const bf16x8 A = __builtin_bit_cast(bf16x8, av);
            const int cs = c - stage * cps;
#pragma unroll
            for (int dt = 0; dt < DTMAX; ++dt) {
                if (dt >= DT) break;
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
            if (dt >= DT) break;
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

// Long rows (Lk > 32 * 20): the same arithmetic, with the logits re-read in
// each pass instead of held in registers.
template <bool FUSED>
__global__ __launch_bounds__(kBlock) void lis_kernel_stream(LisArgs a, LisLaunch p) {
    extern __shared__ uint16_t vt[];
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
    const int nc = (Lk + 31) >> 5;
    const bool active = i0 < a.Lq;
    if (!FUSED && !active) return;

    const int i = min(i0 + r, a.Lq - 1);
    const int32_t* row = a.logits + (g * a.Lq + i) * (int64_t)Lk;
    const int32_t* brow = a.bias ? a.bias + ((g % a.Hb) * a.Lq + i) * (int64_t)Lk : nullptr;
    const int8_t* vg = FUSED ? a.v + g * (int64_t)Lk * a.d : nullptr;
    const LisConsts k = a.k;

    int mx = INT_MIN;
    for (int c = 0; c < nc; ++c) {
        int lg[8];
        load_chunk(lg, row, brow, c, kg, Lk);
#pragma unroll
        for (int t = 0; t < 8; ++t) mx = max(mx, lg[t]);
    }
    mx = max(mx, __shfl_xor(mx, 16, 64));
    mx = max(mx, __shfl_xor(mx, 32, 64));

    uint64_t sum = 0;
    for (int c = 0; c < nc; ++c) {
        int lg[8];
        load_chunk(lg, row, brow, c, kg, Lk);
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            uint64_t s1 = 0;
            iexp_pack(lg[t], mx, k, s1);
            sum += lg[t] != INT_MIN ? s1 : 0;
        }
    }
    sum += __shfl_xor(sum, 16, 64);
    sum += __shfl_xor(sum, 32, 64);
    const uint64_t S2 = sum << 1;

    const int nbytes = (Lk + 1) >> 1;
    const bool row_ok = (i0 + r) < a.Lq;
    uint8_t* crow = a.codes ? a.codes + (g * a.Lq + i) * (int64_t)a.ld_codes : nullptr;
    constexpr int DTMAX = 16;
    const int DT = p.dpad >> 4;
    f32x4 acc[DTMAX];
#pragma unroll
    for (int dt = 0; dt < DTMAX; ++dt) acc[dt] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int cps = p.kb >> 5;
    for (int c = 0; c < nc; ++c) {
        const int stage = c / cps;
        if (FUSED && c % cps == 0) {
            if (c > 0) __syncthreads();
            stage_vt(vt, p.ld, vg, Lk, a.d, p.dpad, stage * p.kb, min(p.kb, nc * 32 - stage * p.kb),
                     a.zp_v, p.dword_ok);
            __syncthreads();
        }
        int lg[8];
        load_chunk(lg, row, brow, c, kg, Lk);
        int code[8];
        uint32_t pbits[8];
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            uint64_t s1 = 0;
            const bool valid = lg[t] != INT_MIN;
            const uint32_t pk = iexp_pack(valid ? lg[t] : mx, mx, k, s1);
            const int cd = lis_code(pk, S2, k);
            code[t] = valid ? cd : 0;
            pbits[t] = valid ? (uint32_t)(127 + k.top - cd) << 7 : 0u;
        }
        if (crow && row_ok) store_codes(crow, nbytes, c, kg, code);
        if (FUSED) {
            u32x4 av;
            av.x = pbits[0] | (pbits[1] << 16);
            av.y = pbits[2] | (pbits[3] << 16);
            av.z = pbits[4] | (pbits[5] << 16);
            av.w = pbits[6] | (pbits[7] << 16);
            const bf16x8 A = __builtin_bit_cast(bf16x8, av);
            const int cs = c - stage * cps;
            for (int dt = 0; dt < DT; ++dt) {
                const u32x4 bv = *reinterpret_cast<const u32x4*>(
                    vt + (16 * dt + r) * p.ld + 32 * cs + 8 * kg);
                acc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, __builtin_bit_cast(bf16x8, bv),
                                                                  acc[dt], 0, 0, 0);
            }
        }
    }

    if (FUSED && active) {
        for (int dt = 0; dt < DT; ++dt) {
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

// ---------------------------------------------------------------------------
// Standalone BitShift Attn x V: exact int32 shift-accumulate on the vector ALUs.
// A workgroup owns unit g and `rows` query rows; `tpr` threads share a row,
// each accumulating 16 output columns.  Keys are processed in stages of `kb`:
// V - zp_V as int16 [kb][16 tpr] and the shift amounts as bytes [rows][kb] in LDS.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) void attn_v_shift_kernel(AvArgs a, int tpr, int rows,
                                                              int ntiles, int kb) {
    extern __shared__ int16_t lds16[];
    const int dpad = 16 * tpr;
    int16_t* sv = lds16;                                          // [kb][dpad]
    uint8_t* ssh = reinterpret_cast<uint8_t*>(lds16 + kb * dpad); // [rows][kb]
    const int64_t total = a.G * (int64_t)ntiles;
    const int64_t lb = xcd_remap(blockIdx.x, total);
    const int64_t g = lb / ntiles;
    const int tile = (int)(lb - g * ntiles);
    const int row_local = threadIdx.x / tpr;
    const int cgrp = threadIdx.x - row_local * tpr;
    const int irow = tile * rows + row_local;
    const int Lk = a.Lk;

    uint32_t acc[16];
#pragma unroll
    for (int q = 0; q < 16; ++q) acc[q] = 0;

    for (int k0 = 0; k0 < Lk; k0 += kb) {
        const int kc = min(kb, Lk - k0);
        __syncthreads();
        for (int idx = threadIdx.x; idx < kb * dpad; idx += blockDim.x) {
            const int jj = idx / dpad;
            const int dd = idx - jj * dpad;
            const int j = k0 + jj;
            sv[idx] = (jj < kc && dd < a.d) ? (int16_t)((int)a.v[(g * Lk + j) * (int64_t)a.d + dd] - a.zp_v)
                                            : (int16_t)0;
        }
        for (int idx = threadIdx.x; idx < rows * kb; idx += blockDim.x) {
            const int rl = idx / kb;
            const int jj = idx - rl * kb;
            const int ir = tile * rows + rl;
            const int j = k0 + jj;
            int sh = 0;
            if (ir < a.Lq && jj < kc) {
                const uint8_t byte = a.codes[(g * a.Lq + ir) * (int64_t)a.ld_codes + (j >> 1)];
                const int code = (j & 1) ? (byte >> 4) : (byte & 15);
                sh = a.top - code;
            }
            ssh[idx] = (uint8_t)sh;
        }
        __syncthreads();
        if (irow < a.Lq) {
            const int16_t* vbase = sv + 16 * cgrp;
            const uint8_t* srow = ssh + row_local * kb;
            for (int jj = 0; jj < kc; ++jj) {
                const int sh = srow[jj];
                const int16_t* vr = vbase + jj * dpad;
#pragma unroll
                for (int q = 0; q < 16; ++q) acc[q] += (uint32_t)(int32_t)vr[q] << sh;
            }
        }
    }
    if (irow < a.Lq) {
        int32_t* orow = a.out + (g * a.Lq + irow) * (int64_t)a.d;
#pragma unroll
        for (int q = 0; q < 16; ++q) {
            const int col = 16 * cgrp + q;
            if (col < a.d) orow[col] = (int32_t)acc[q];
        }
    }
}

template <int NC>
hipError_t launch_nc(const LisArgs& a, const LisLaunch& p, dim3 grid, size_t lds, bool fused,
                     hipStream_t stream) {
    const int DT = p.dpad >> 4;
    if (!fused)
        hipLaunchKernelGGL((lis_kernel<NC, false, 1>), grid, dim3(kBlock), 0, stream, a, p);
    else if (DT <= 2)
        hipLaunchKernelGGL((lis_kernel<NC, true, 2>), grid, dim3(kBlock), lds, stream, a, p);
    else if (DT <= 4)
        hipLaunchKernelGGL((lis_kernel<NC, true, 4>), grid, dim3(kBlock), lds, stream, a, p);
    else
        hipLaunchKernelGGL((lis_kernel<NC, true, 16>), grid, dim3(kBlock), lds, stream, a, p);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_lis(const LisArgs& a, hipStream_t stream) {
    const bool fused = a.out != nullptr;
    LisLaunch p;
    p.ntiles = (a.Lq + kRowsPerBlock - 1) / kRowsPerBlock;
    const int nc = (a.Lk + 31) / 32;
    p.dpad = fused ? 16 * ((a.d + 15) / 16) : 16;
    // V^T stage: at most 40 KB of LDS so that several workgroups share a CU.
    const int max_keys = (40960 / (2 * p.dpad) - 8) / 32 * 32;
    p.kb = std::max(32, std::min(nc * 32, max_keys));
    p.ld = p.kb + 8;
    p.dword_ok = (a.d % 4 == 0) && ((reinterpret_cast<uintptr_t>(a.v) & 3) == 0);
    const size_t lds = fused ? (size_t)p.dpad * p.ld * sizeof(uint16_t) : 0;
    const int64_t blocks = a.G * (int64_t)p.ntiles;
    const dim3 grid((unsigned)blocks);
    if (nc <= 2) return launch_nc<2>(a, p, grid, lds, fused, stream);
    if (nc <= 4) return launch_nc<4>(a, p, grid, lds, fused, stream);
    if (nc <= 7) return launch_nc<7>(a, p, grid, lds, fused, stream);
    if (nc <= 12) return launch_nc<12>(a, p, grid, lds, fused, stream);
    if (nc <= 20) return launch_nc<20>(a, p, grid, lds, fused, stream);
    if (fused)
        hipLaunchKernelGGL((lis_kernel_stream<true>), grid, dim3(kBlock), lds, stream, a, p);
    else
        hipLaunchKernelGGL((lis_kernel_stream<false>), grid, dim3(kBlock), 0, stream, a, p);
    return hipGetLastError();
}

hipError_t launch_attn_v_shift(const AvArgs& a, hipStream_t stream) {
    int tpr = 1;
    while (16 * tpr < a.d) tpr <<= 1;          // threads per row, 16 columns each
    const int rows = kBlock / tpr;
    const int ntiles = (a.Lq + rows - 1) / rows;
    const int dpad = 16 * tpr;
    // LDS: kb * dpad int16 + rows * kb bytes <= 32 KB
    int kb = 32768 / (2 * dpad + rows);
    kb = std::max(16, std::min(kb, 256));
    const size_t lds = (size_t)kb * dpad * sizeof(int16_t) + (size_t)rows * kb;
    const int64_t blocks = a.G * (int64_t)ntiles;
    hipLaunchKernelGGL(attn_v_shift_kernel, dim3((unsigned)blocks), dim3(kBlock), lds, stream, a,
                       tpr, rows, ntiles, kb);
    return hipGetLastError();
}

}  // namespace fqvit
