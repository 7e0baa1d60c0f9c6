// Integer-only attention from int8 Q and K for long rows (8 to 20 chunks of
// 32 keys, up to 640 keys) on gfx950: the integer GEMM Q K^T of Sec. 3.1 on
// MFMA, Log-Int-Softmax (Supplement A.2, Alg. 1 and 2) and the BitShift
// Attn x V of Sec. 3.3, logits and codes never leaving the chip.
//
// One workgroup of kQkLongWaves wavefronts per unit stages V^T (bf16), K
// (int8, XOR-swizzled as in lis_qk_kernel.h) and each key's zero-point term
// in LDS once.  A row of several hundred keys does not fit a lane's registers,
// and its logits cost two MFMAs per 32-key chunk from LDS, so each 16-query
// tile makes three passes over the keys, recomputing the logits in each: the
// row maximum, the exact I-Exp sum, and the codes with the product P V.  The
// chunk count is a run-time value (the work of one chunk is unrolled); the
// last chunk's keys past Lk get P = 0 and meet the padding of V^T.
#include "lis_long.h"
#include "lis_qk_kernel.h"

namespace fqvit {
namespace lis {

constexpr int kQkLongWaves = 12;
constexpr int kQkLongBlock = 64 * kQkLongWaves;

// Logits of chunk c for lane (query r, group kg): keys 32 c + 4 kg + t
// (t < 4) and 32 c + 16 + 4 kg + (t - 4), INT_MIN past Lk; the bias row (if
// any) added.
template <int DK>
__device__ __forceinline__ void qk_long_chunk(int (&lg)[8], const int8_t* kst, const int32_t* ck,
                                              const i32x4v (&qb)[DK >= 64 ? DK / 64 : 1],
                                              int64_t qb8, const int32_t* brow, int c, int r, int kg,
                                              int Lk) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int kt = 2 * c + h;
        const int key = 16 * kt + r;
        const int j0 = 16 * kt + 4 * kg;
        // the per-key zero-point terms as the initial accumulator
        i32x4v s = *reinterpret_cast<const i32x4v*>(ck + j0);
        if constexpr (DK >= 64) {
#pragma unroll
            for (int m = 0; m < DK / 64; ++m) {
                const i32x4v av = *reinterpret_cast<const i32x4v*>(kst + kst_off<DK>(key, 4 * m + kg));
                s = __builtin_amdgcn_mfma_i32_16x16x64_i8(av, qb[m], s, 0, 0, 0);
            }
        } else {
            const int64_t av = *reinterpret_cast<const int64_t*>(kst + key * DK + 8 * kg);
            s = __builtin_amdgcn_mfma_i32_16x16x32_i8(av, qb8, s, 0, 0, 0);
        }
#pragma unroll
        for (int t = 0; t < 4; ++t) lg[4 * h + t] = j0 + t < Lk ? s[t] : INT_MIN;
    }
    if (brow) {
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            const int j = 32 * c + 4 * kg + (t < 4 ? t : 12 + t);
            if (j < Lk) lg[t] += brow[j];
        }
    }
}

template <int DTMAX, bool FP, int DK, bool P0 = false>
__global__ __launch_bounds__(kQkLongBlock) void lis_qk_long_kernel(LisArgs a, QkArgs qa,
                                                                   LisLaunch p) {
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    const int nc = (a.Lk + 31) >> 5;
    const int kp = 32 * nc;                       // staged keys (zero past Lk)
    uint16_t* vt = reinterpret_cast<uint16_t*>(smem);
    int8_t* kst = reinterpret_cast<int8_t*>(smem + p.vt_bytes);
    int32_t* ck = reinterpret_cast<int32_t*>(smem + p.vt_bytes + kp * DK);
    const int64_t g = blockIdx.x;
    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const int r = lane & 15;
    const int kg = lane >> 4;
    const int Lk = a.Lk;

    LisConsts k = a.k;
    k.u_max &= 0xFFFFFFu;
    k.d_ln2 &= 0xFFFFFFu;
    k.magic &= 0xFFFFFFu;

    // V^T, K and the per-key zero-point terms of the unit
    long_stage_vt<DTMAX, kQkLongBlock>(vt, p.ld, a.v + g * (int64_t)Lk * a.d, Lk, a.d, kp, a.zp_v,
                                       p.vec_ok);
    const int8_t* kg_base = qa.k + g * (int64_t)Lk * DK;
    for (int w = threadIdx.x; w < kp * (DK / 16); w += kQkLongBlock) {
        const int j = w / (DK / 16);
        const int u = w - j * (DK / 16);
        i32x4v val = {0, 0, 0, 0};
        if (j < Lk) val = *reinterpret_cast<const i32x4v*>(kg_base + (int64_t)j * DK + 16 * u);
        *reinterpret_cast<i32x4v*>(kst + kst_off<DK>(j, u)) = val;
    }
    __syncthreads();
    for (int j = threadIdx.x; j < kp; j += kQkLongBlock) {
        int s = 0;
#pragma unroll
        for (int u = 0; u < DK / 16; ++u) {
            const i32x4v v = *reinterpret_cast<const i32x4v*>(kst + kst_off<DK>(j, u));
            s = __builtin_amdgcn_sdot4(v.x, 0x01010101, s, false);
            s = __builtin_amdgcn_sdot4(v.y, 0x01010101, s, false);
            s = __builtin_amdgcn_sdot4(v.z, 0x01010101, s, false);
            s = __builtin_amdgcn_sdot4(v.w, 0x01010101, s, false);
        }
        ck[j] = -(qa.zq * s);     // the per-key zero-point term, stored negated
    }
    __syncthreads();

    const int8_t* q_base = qa.q + g * (int64_t)a.Lq * DK;
    const int32_t* bplane = a.bias ? a.bias + (g % a.Hb) * (int64_t)a.Lq * Lk : nullptr;
    const uint32_t kr = ((uint32_t)(k.top + 1) << 25) - 1u;
    const int ptop = (127 + k.top) << 7;

    for (int tile = wave; tile < p.ntiles; tile += kQkLongWaves) {
        const int i0 = 16 * tile;
        const int i = min(i0 + r, a.Lq - 1);
        const int8_t* qrow = q_base + (int64_t)i * DK;
        i32x4v qb[DK >= 64 ? DK / 64 : 1];
        int64_t qb8 = 0;
        if constexpr (DK >= 64) {
#pragma unroll
            for (int m = 0; m < DK / 64; ++m)
                qb[m] = *reinterpret_cast<const i32x4v*>(qrow + 64 * m + 16 * kg);
        } else {
            qb[0] = i32x4v{0, 0, 0, 0};
            qb8 = *reinterpret_cast<const int64_t*>(qrow + 8 * kg);
        }
        const int32_t* brow = bplane ? bplane + (int64_t)i * Lk : nullptr;

        int mx = INT_MIN;
#pragma unroll 1
        for (int c = 0; c < nc; ++c) {
            int lg[8];
            qk_long_chunk<DK>(lg, kst, ck, qb, qb8, brow, c, r, kg, Lk);
#pragma unroll
            for (int t = 0; t < 8; ++t) mx = max(mx, lg[t]);
        }
        mx = row4_max(mx);

        RowState st;
        if constexpr (FP) {
            double part[2] = {0.0, 0.0};
#pragma unroll 1
            for (int c = 0; c < nc; ++c) {
                int lg[8];
                qk_long_chunk<DK>(lg, kst, ck, qb, qb8, brow, c, r, kg, Lk);
#pragma unroll
                for (int t = 0; t < 8; ++t) {
                    const float e = iexp_f<P0>(lg[t], mx, k);
                    part[t & 1] += lg[t] != INT_MIN ? (double)e : 0.0;
                }
            }
            const double S2 = 2.0 * row4_sum(part[0] + part[1]);
            st.S2s = S2 * kCodeScale;
            st.sc = kCodeScale;
            asm volatile("" : "+s"(st.sc));
            st.tau = third_floor_f32(S2);
        } else {
            uint64_t sum = 0;
#pragma unroll 1
            for (int c = 0; c < nc; ++c) {
                int lg[8];
                qk_long_chunk<DK>(lg, kst, ck, qb, qb8, brow, c, r, kg, Lk);
#pragma unroll
                for (int t = 0; t < 8; ++t) {
                    uint32_t z;
                    const uint32_t qL = iexp_qL(lg[t], mx, k, z);
                    sum += lg[t] != INT_MIN ? ((uint64_t)qL << (k.n - (int)z)) : 0ull;
                }
            }
            st.rs = row_sum(sum, k);
        }

        f32x4 acc[DTMAX];
#pragma unroll
        for (int dt = 0; dt < DTMAX; ++dt) acc[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll 1
        for (int c = 0; c < nc; ++c) {
            int lg[8];
            qk_long_chunk<DK>(lg, kst, ck, qb, qb8, brow, c, r, kg, Lk);
            uint32_t pbits[8];
#pragma unroll
            for (int t = 0; t < 8; ++t) {
                const bool valid = lg[t] != INT_MIN;
                if constexpr (FP) {
                    const int eb = __float_as_int(iexp_f<P0>(valid ? lg[t] : mx, mx, k));
                    pbits[t] = valid ? (127u + code_rev_f(eb, st, kr)) << 7 : 0u;
                } else {
                    uint32_t z;
                    const uint32_t qL = iexp_qL(valid ? lg[t] : mx, mx, k, z);
                    const int cd = lis_code(qL, z, st.rs, k);
                    pbits[t] = valid ? (uint32_t)(ptop - (cd << 7)) : 0u;
                }
            }
            const u32x4 pb = {pbits[0] | (pbits[1] << 16), pbits[2] | (pbits[3] << 16),
                              pbits[4] | (pbits[5] << 16), pbits[6] | (pbits[7] << 16)};
            chunk_mfma<DTMAX, false, true>(acc, pb, vt, p.ld, c, r, kg);
        }
        store_out_t<DTMAX>(acc, a, g, i0, r, kg, p.out_vec);
    }
}

template <int DK>
hipError_t launch_qk_long_dk(int dtm, int fpm, const LisArgs& a, const QkArgs& qa,
                             const LisLaunch& p, size_t lds, hipStream_t stream) {
    const dim3 grid((unsigned)a.G), block(kQkLongBlock);
#define FQ_QKL(DT, F, P0) \
    launch_kernel(lis_qk_long_kernel<DT, F, DK, P0>, grid, block, lds, stream, a, qa, p)
    if (dtm == 2) {
        if (fpm == 2) FQ_QKL(2, true, true);
        else if (fpm == 1) FQ_QKL(2, true, false);
        else FQ_QKL(2, false, false);
    } else {
        if (fpm == 2) FQ_QKL(4, true, true);
        else if (fpm == 1) FQ_QKL(4, true, false);
        else FQ_QKL(4, false, false);
    }
#undef FQ_QKL
    return hipGetLastError();
}

hipError_t launch_qk_long(int dk, int dtm, int fp, const LisArgs& a, const QkArgs& qa,
                          const LisLaunch& p, size_t lds, hipStream_t stream) {
    return dk == 32 ? launch_qk_long_dk<32>(dtm, fp, a, qa, p, lds, stream)
                    : launch_qk_long_dk<64>(dtm, fp, a, qa, p, lds, stream);
}

}  // namespace lis
}  // namespace fqvit
