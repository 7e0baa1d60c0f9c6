// Integer-only multi-head self-attention from int8 queries and keys on gfx950:
// the MinMax-quantized MatMul of Sec. 3.1 (Q K^T as an integer GEMM) feeding
// Log-Int-Softmax and the BitShift Attn x V of Sec. 3.3 (the dataflow of its
// Fig. 4), with the logits never leaving the chip.
//
// One workgroup per attention unit (as in the unit kernel of lis_device.h):
// V^T is staged once in LDS as bf16, K once as int8 with each key's zero-point
// term, and each wavefront walks the unit's 16-query tiles.  For a tile, its
// queries' bytes are the B operand of v_mfma_i32_16x16x{64,32}_i8 and 16 keys
// of K the A operand, so one MFMA gives S^T for 16 keys x 16 queries with lane
// (query r, group kg) holding keys 4 kg .. 4 kg + 3 of the key tile: two key
// tiles make exactly the 8 keys per 32-key chunk that the Log-Int-Softmax
// code of lis_device.h keeps per lane.  Both operands take contiguous bytes of
// the feature dimension in the same lane order, so the dot product covers
// every feature once whatever order the instruction uses inside a lane group.
//
// With zero points (int8 containers; the 2^(b-1) offset cancels):
//   sum_c (q - zq)(k - zk) = S - zk sum_c q - zq sum_c k + dk zq zk,
// S = sum_c q k from the MFMA; the per-key term zq sum_c k is computed once per
// unit (stored negated) and added to S.  The per-query term dk zq zk - zk
// sum_c q is left out: it is the same for every key of a row, and the
// Log-Int-Softmax of a row depends only on the differences of its logits
// (I-Exp takes max - v).  All sums are exact in int32 (|S| <= dk 255^2 < 2^24
// for dk <= 256).
#pragma once

#include "lis_device.h"

namespace fqvit {
namespace lis {

struct QkArgs {
    const int8_t* q;    // [G, Lq, DK] int8 container
    const int8_t* k;    // [G, Lk, DK] int8 container
    int32_t zq;         // zero point of q, container form
    int32_t zk;         // zero point of k: carried, not used (it cancels, see above)
};

typedef int32_t i32x4v __attribute__((ext_vector_type(4)));

// Byte offset of 16-byte unit u of key j in the staged K (DK bytes per key).
// For DK >= 64 the units are XOR-swizzled with bits 2..3 of the key so that
// the 16 keys read by one lane group fall on distinct LDS banks.
template <int DK>
__device__ __forceinline__ int kst_off(int j, int u) {
    if constexpr (DK >= 64) return j * DK + 16 * (u ^ ((j >> 2) & 3));
    return j * DK + 16 * u;
}

template <int NC, int DTMAX, bool HALF, bool FP, int DK, bool P0 = false>
__global__ __launch_bounds__(kBlock, 3) void lis_qk_kernel(LisArgs a, QkArgs qa, LisLaunch p) {
    constexpr int NT = HALF ? 4 : 8;
    constexpr int KP = 32 * NC;                 // staged keys (zero past Lk)
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    uint16_t* vt = reinterpret_cast<uint16_t*>(smem);
    int8_t* kst = reinterpret_cast<int8_t*>(smem + p.vt_bytes);
    int32_t* ck = reinterpret_cast<int32_t*>(smem + p.vt_bytes + KP * DK);
    const int64_t g = blockIdx.x;
    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const int r = lane & 15;
    const int kg = lane >> 4;

    LisConsts k = a.k;
    k.u_max &= 0xFFFFFFu;
    k.d_ln2 &= 0xFFFFFFu;
    k.magic &= 0xFFFFFFu;

    // V^T and K of the unit into LDS
    StageRegs sr;
    stage_load(sr, a.v + g * (int64_t)a.Lk * a.d, a.Lk, a.d, DTMAX, 0, KP, p.vec_ok);
    const int8_t* kg_base = qa.k + g * (int64_t)a.Lk * DK;
    for (int w = threadIdx.x; w < KP * (DK / 16); w += kBlock) {
        const int j = w / (DK / 16);
        const int u = w - j * (DK / 16);
        i32x4v val = {0, 0, 0, 0};
        if (j < a.Lk) val = *reinterpret_cast<const i32x4v*>(kg_base + (int64_t)j * DK + 16 * u);
        *reinterpret_cast<i32x4v*>(kst + kst_off<DK>(j, u)) = val;
    }
    stage_store(sr, vt, p.ld, DTMAX, KP, a.zp_v);
    __syncthreads();
    // per-key zero-point term zq sum_c k[j][c] (0 for padded keys, whose
    // logits are masked anyway)
    if (threadIdx.x < KP) {
        const int j = threadIdx.x;
        int s = 0;
#pragma unroll
        for (int u = 0; u < DK / 16; ++u) {
            const i32x4v v = *reinterpret_cast<const i32x4v*>(kst + kst_off<DK>(j, u));
            s = __builtin_amdgcn_sdot4(v.x, 0x01010101, s, false);
            s = __builtin_amdgcn_sdot4(v.y, 0x01010101, s, false);
            s = __builtin_amdgcn_sdot4(v.z, 0x01010101, s, false);
            s = __builtin_amdgcn_sdot4(v.w, 0x01010101, s, false);
        }
        ck[j] = -(qa.zq * s);        // stored negated: the initial accumulator of the logits
    }
    __syncthreads();

    const int8_t* q_base = qa.q + g * (int64_t)a.Lq * DK;
    const int32_t* bplane = a.bias ? a.bias + (g % a.Hb) * (int64_t)a.Lq * a.Lk : nullptr;

    // B operand: this lane's bytes of query row i (DK / 4 bytes)
    i32x4v qb[DK >= 64 ? DK / 64 : 1];
    int64_t qb8 = 0;
    auto load_q = [&](int t, i32x4v (&dst)[DK >= 64 ? DK / 64 : 1], int64_t& dst8) {
        const int8_t* qrow = q_base + (int64_t)min(16 * t + r, a.Lq - 1) * DK;
        if constexpr (DK >= 64) {
#pragma unroll
            for (int m = 0; m < DK / 64; ++m)
                dst[m] = *reinterpret_cast<const i32x4v*>(qrow + 64 * m + 16 * kg);
        } else {
            dst8 = *reinterpret_cast<const int64_t*>(qrow + 8 * kg);
        }
    };
    int tile = (wave + (int)(g & 3)) & 3;
    if (tile < p.ntiles) load_q(tile, qb, qb8);
    for (; tile < p.ntiles; tile += 4) {
        const int i0 = 16 * tile;
        const int i = min(i0 + r, a.Lq - 1);

        // logits of this tile in the Log-Int-Softmax lane layout
        int lg[NC][8];
#pragma unroll
        for (int c = 0; c < NC; ++c) {
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                if (HALF && c == NC - 1 && h == 1) {
#pragma unroll
                    for (int t = 4; t < 8; ++t) lg[c][t] = INT_MIN;
                    continue;
                }
                const int kt = 2 * c + h;
                const int key = 16 * kt + r;          // A operand row of this lane
                const int j0 = 16 * kt + 4 * kg;      // keys of s[0..3]
                // the per-key zero-point terms enter as the accumulator's
                // initial value (same layout: lane (r, kg) holds keys j0 ..
                // j0 + 3), so the sum needs no separate add
                i32x4v s = *reinterpret_cast<const i32x4v*>(ck + j0);
                if constexpr (DK >= 64) {
#pragma unroll
                    for (int m = 0; m < DK / 64; ++m) {
                        const i32x4v av =
                            *reinterpret_cast<const i32x4v*>(kst + kst_off<DK>(key, 4 * m + kg));
                        s = __builtin_amdgcn_mfma_i32_16x16x64_i8(av, qb[m], s, 0, 0, 0);
                    }
                } else {
                    const int64_t av = *reinterpret_cast<const int64_t*>(kst + key * DK + 8 * kg);
                    s = __builtin_amdgcn_mfma_i32_16x16x32_i8(av, qb8, s, 0, 0, 0);
                }
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    // the per-query term zp_q zp_k dk - zp_k sum_c q[i][c] is
                    // left out: the Log-Int-Softmax of a row depends only on
                    // the differences of its logits (u = max - v)
                    const int v = s[t];
                    // only the last chunk can hold keys past Lk
                    lg[c][4 * h + t] = (c < NC - 1 || j0 + t < a.Lk) ? v : INT_MIN;
                }
            }
        }
        // the next tile's query bytes, in flight during the rest of this tile
        load_q(tile + 4 < p.ntiles ? tile + 4 : tile, qb, qb8);
        if (bplane) {   // uniform: the bias of the lane's row, in a pass of its own
            const int32_t* brow = bplane + (int64_t)i * a.Lk;
#pragma unroll
            for (int c = 0; c < NC; ++c) {
#pragma unroll
                for (int t = 0; t < 8; ++t) {
                    const int j = 32 * c + 4 * kg + (t < 4 ? t : 12 + t);
                    if (c < NC - 1 || j < a.Lk) lg[c][t] += brow[j];
                }
            }
        }
        uint32_t zb[NC][2];
        const RowState st = tile_iexp<NC, FP, NT, P0>(lg, zb, k);
        f32x4 acc[DTMAX];
#pragma unroll
        for (int dt = 0; dt < DTMAX; ++dt) acc[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            const u32x4 pb = chunk_pbits<NC, FP, NT>(lg, zb, st, k, c);
            if (HALF && c == NC - 1)
                chunk_mfma<DTMAX, true, true>(acc, pb, vt, p.ld, c, r, kg);
            else
                chunk_mfma<DTMAX, false, true>(acc, pb, vt, p.ld, c, r, kg);
            __builtin_amdgcn_sched_barrier(0);
        }
        store_out_t<DTMAX>(acc, a, g, i0, r, kg, p.out_vec);
    }
}

// fpm: 0 the integer path, 1 the float path, 2 the float path with the
// I-Exp pre-shift 0.
template <int DK, int NC>
hipError_t launch_qk_nc(int dtm, bool half, int fpm, const LisArgs& a, const QkArgs& qa,
                        const LisLaunch& p, size_t lds, hipStream_t stream) {
    const dim3 grid((unsigned)a.G), block(kBlock);
#define FQ_QK(DT, H, F, P0) \
    launch_kernel(lis_qk_kernel<NC, DT, H, F, DK, P0>, grid, block, lds, stream, a, qa, p)
#define FQ_QK_F(DT, H) \
    if (fpm == 2) FQ_QK(DT, H, true, true); else if (fpm == 1) FQ_QK(DT, H, true, false); \
    else FQ_QK(DT, H, false, false)
#define FQ_QK_H(DT) \
    if (half) { FQ_QK_F(DT, true); } else { FQ_QK_F(DT, false); }
    if (dtm == 2) { FQ_QK_H(2) }
    else { FQ_QK_H(4) }
#undef FQ_QK_H
#undef FQ_QK_F
#undef FQ_QK
    return hipGetLastError();
}

template <int DK>
hipError_t launch_qk_dk(int nc, int dtm, bool half, int fp, const LisArgs& a, const QkArgs& qa,
                        const LisLaunch& p, size_t lds, hipStream_t stream) {
    switch (nc) {
        case 1: return launch_qk_nc<DK, 1>(dtm, half, fp, a, qa, p, lds, stream);
        case 2: return launch_qk_nc<DK, 2>(dtm, half, fp, a, qa, p, lds, stream);
        case 3: return launch_qk_nc<DK, 3>(dtm, half, fp, a, qa, p, lds, stream);
        case 4: return launch_qk_nc<DK, 4>(dtm, half, fp, a, qa, p, lds, stream);
        case 5: return launch_qk_nc<DK, 5>(dtm, half, fp, a, qa, p, lds, stream);
        case 6: return launch_qk_nc<DK, 6>(dtm, half, fp, a, qa, p, lds, stream);
        case 7: return launch_qk_nc<DK, 7>(dtm, half, fp, a, qa, p, lds, stream);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_qk_dk32(int nc, int dtm, bool half, int fp, const LisArgs& a, const QkArgs& qa,
                          const LisLaunch& p, size_t lds, hipStream_t stream);
// Rows of 8 to 20 chunks (lis_qk_long.hip): one workgroup of 12 wavefronts per
// unit, three passes over K in LDS per tile.
hipError_t launch_qk_long(int dk, int dtm, int fp, const LisArgs& a, const QkArgs& qa,
                          const LisLaunch& p, size_t lds, hipStream_t stream);
hipError_t launch_qk_dk64(int nc, int dtm, bool half, int fp, const LisArgs& a, const QkArgs& qa,
                          const LisLaunch& p, size_t lds, hipStream_t stream);

}  // namespace lis
}  // namespace fqvit
