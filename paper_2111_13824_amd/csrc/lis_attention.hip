// Log-Int-Softmax attention for gfx950: launch selection, the long-row
// streaming kernel and the standalone BitShift Attn x V kernel.  The register
// kernels (lis_device.h) are instantiated per chunk count in lis_inst_*.hip.
#include "lis_long.h"

namespace fqvit {
namespace lis {

// Long rows, head dimensions above 64 and fused calls that also write the
// codes: the same arithmetic with the logits re-read in each pass instead of
// held in registers.  DTMAX = dpad / 16 output column tiles (1 without the
// product), a template constant so that the accumulators stay in registers.
// FP: the float path of the unit kernel (binary32 e, binary64 row sum and the
// funnel-shift code), for scales where it is exact; else the integer path.
template <bool FUSED, int DTMAX, bool FP>
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
    LisConsts k = a.k;
    k.d_ln2 &= 0xFFFFFFu;
    k.magic &= 0xFFFFFFu;

    const int i = min(i0 + r, a.Lq - 1);
    const int64_t roff = (g * a.Lq + i) * (int64_t)Lk;
    const int32_t* row = a.logits + roff;
    const int64_t boff = a.bias ? ((g % a.Hb) * a.Lq + i) * (int64_t)Lk : 0;
    const int32_t* brow = a.bias ? a.bias + boff : nullptr;
    const int8_t* vg = FUSED ? a.v + g * (int64_t)Lk * a.d : nullptr;
    const bool tail_vec = roff + 32 * nc <= p.n_logits && (!brow || boff + 32 * nc <= p.n_bias);

    int mx = INT_MIN;
    for (int c = 0; c < nc; ++c) {
        int lg[8];
        load_chunk<false>(lg, row, brow, c, kg, Lk, tail_vec);
#pragma unroll
        for (int t = 0; t < 8; ++t) mx = max(mx, lg[t]);
    }
    mx = row4_max(mx);

    RowState st;
    if constexpr (FP) {
        // two partial sums of integers below 2^53: exact in any order
        double part[2] = {0.0, 0.0};
        for (int c = 0; c < nc; ++c) {
            int lg[8];
            load_chunk<false>(lg, row, brow, c, kg, Lk, tail_vec);
#pragma unroll
            for (int t = 0; t < 8; ++t) {
                const float e = iexp_f(lg[t], mx, k);
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
        for (int c = 0; c < nc; ++c) {
            int lg[8];
            load_chunk<false>(lg, row, brow, c, kg, Lk, tail_vec);
#pragma unroll
            for (int t = 0; t < 8; ++t) {
                uint32_t z;
                const uint32_t qL = iexp_qL(lg[t], mx, k, z);
                sum += lg[t] != INT_MIN ? ((uint64_t)qL << (k.n - (int)z)) : 0ull;
            }
        }
        st.rs = row_sum(sum, k);
    }
    const uint32_t kr = ((uint32_t)(k.top + 1) << 25) - 1u;

    const bool row_ok = (i0 + r) < a.Lq;
    uint8_t* crow = a.codes ? a.codes + (g * a.Lq + i) * (int64_t)a.ld_codes : nullptr;
    f32x4 acc[DTMAX];
#pragma unroll
    for (int dt = 0; dt < DTMAX; ++dt) acc[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int ptop = (127 + k.top) << 7;
    const int cps = p.kb >> 5;
    for (int c = 0; c < nc; ++c) {
        const int stage = c / cps;
        if (FUSED && c % cps == 0) {
            if (c > 0) __syncthreads();
            stage_vt(vt, p.ld, vg, Lk, a.d, p.ncg, stage * p.kb,
                     min(p.kb, nc * 32 - stage * p.kb), a.zp_v, p.vec_ok);
            __syncthreads();
        }
        int lg[8];
        load_chunk<false>(lg, row, brow, c, kg, Lk, tail_vec);
        int code[8];
        uint32_t pbits[8];
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            const bool valid = lg[t] != INT_MIN;
            if constexpr (FP) {
                const int eb = __float_as_int(iexp_f(valid ? lg[t] : mx, mx, k));
                code[t] = 0;
                if (!FUSED || crow) code[t] = valid ? code_f(eb, st, k.top) : 0;
                pbits[t] = (FUSED && valid) ? (127u + code_rev_f(eb, st, kr)) << 7 : 0u;
            } else {
                uint32_t z;
                const uint32_t qL = iexp_qL(valid ? lg[t] : mx, mx, k, z);
                const int cd = lis_code(qL, z, st.rs, k);
                code[t] = valid ? cd : 0;
                pbits[t] = valid ? (uint32_t)(ptop - (cd << 7)) : 0u;
            }
        }
        if (crow && row_ok) store_codes_row(crow, Lk, k.top, c, kg, code);
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
                const u32x4 bv = *reinterpret_cast<const u32x4*>(
                    vt + (16 * dt + r) * p.ld + 32 * cs + 8 * kg);
                acc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, __builtin_bit_cast(bf16x8, bv),
                                                                  acc[dt], 0, 0, 0);
            }
        }
    }

    if (FUSED && active) {
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

// The same product for codes of any width b (bytes for b >= 5) at the output
// scale s_V / 2^W, W = min(2^b - 1, 44): each term is (V - zp_V) 2^(W - code),
// exact in int64, or for a code above W (never one from Log-Int-Softmax) the
// arithmetic right shift of V - zp_V by code - W, i.e. its floor.  Sums are
// accumulated modulo 2^64.  Layout and staging as attn_v_shift_kernel, with
// the codes themselves staged as bytes.
__global__ __launch_bounds__(kBlock) void attn_v_shift_wide_kernel(AvWideArgs a, int tpr, int rows,
                                                                   int ntiles, int kb) {
    extern __shared__ int16_t lds16[];
    const int dpad = 16 * tpr;
    int16_t* sv = lds16;                                            // [kb][dpad]
    uint8_t* scode = reinterpret_cast<uint8_t*>(lds16 + kb * dpad); // [rows][kb]
    const int64_t total = a.G * (int64_t)ntiles;
    const int64_t lb = xcd_remap(blockIdx.x, total);
    const int64_t g = lb / ntiles;
    const int tile = (int)(lb - g * ntiles);
    const int row_local = threadIdx.x / tpr;
    const int cgrp = threadIdx.x - row_local * tpr;
    const int irow = tile * rows + row_local;
    const int Lk = a.Lk;

    uint64_t acc[16];
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
            int code = a.W;     // padding keys: any code (their V is 0)
            if (ir < a.Lq && jj < kc) {
                const uint8_t* crow = a.codes + (g * a.Lq + ir) * (int64_t)a.ld_codes;
                if (a.bits <= 4) {
                    const uint8_t byte = crow[j >> 1];
                    code = (j & 1) ? (byte >> 4) : (byte & 15);
                } else {
                    code = crow[j];
                }
            }
            scode[idx] = (uint8_t)code;
        }
        __syncthreads();
        if (irow < a.Lq) {
            const int16_t* vbase = sv + 16 * cgrp;
            const uint8_t* srow = scode + row_local * kb;
            for (int jj = 0; jj < kc; ++jj) {
                const int code = srow[jj];
                const int16_t* vr = vbase + jj * dpad;
                if (code <= a.W) {
                    const int sh = a.W - code;
#pragma unroll
                    for (int q = 0; q < 16; ++q) acc[q] += (uint64_t)(int64_t)vr[q] << sh;
                } else {
                    const int sh = min(code - a.W, 63);
#pragma unroll
                    for (int q = 0; q < 16; ++q) acc[q] += (uint64_t)((int64_t)vr[q] >> sh);
                }
            }
        }
    }
    if (irow < a.Lq) {
        int64_t* orow = a.out + (g * a.Lq + irow) * (int64_t)a.d;
#pragma unroll
        for (int q = 0; q < 16; ++q) {
            const int col = 16 * cgrp + q;
            if (col < a.d) orow[col] = (int64_t)acc[q];
        }
    }
}

}  // namespace lis

namespace {

template <bool FP>
void launch_stream(bool fused, int dt, dim3 grid, size_t lds, hipStream_t stream,
                   const LisArgs& a, const lis::LisLaunch& p) {
    using namespace lis;
    if (!fused)
        launch_kernel(lis_kernel_stream<false, 1, FP>, grid, dim3(kBlock), 0, stream, a, p);
    else if (dt == 2)
        launch_kernel(lis_kernel_stream<true, 2, FP>, grid, dim3(kBlock), lds, stream, a, p);
    else if (dt == 4)
        launch_kernel(lis_kernel_stream<true, 4, FP>, grid, dim3(kBlock), lds, stream, a, p);
    else if (dt == 8)
        launch_kernel(lis_kernel_stream<true, 8, FP>, grid, dim3(kBlock), lds, stream, a, p);
    else
        launch_kernel(lis_kernel_stream<true, 16, FP>, grid, dim3(kBlock), lds, stream, a, p);
}

}  // namespace

// LDS of one workgroup on gfx950.
constexpr size_t kMaxLdsBytes = 160 * 1024;

// Wavefronts per unit of the unit kernel: units of at most four 16-row tiles
// (and rows of at most four chunks, whose V^T 64 threads can stage) get one
// wavefront per tile up to two, so that the per-wavefront set-up serves
// several tiles.  Measured on Swin-S (6144 units of 49 x 49, d = 32): two
// wavefronts per unit 41.4 us, one 43.7 us, four 46.6-47.3 us.
int unit_waves(int nc, int tiles16) {
    if (nc > 4 || tiles16 > 4) return 4;
    return tiles16 == 1 ? 1 : 2;
}

hipError_t launch_lis(const LisArgs& a, hipStream_t stream) {
    using namespace lis;
    const bool fused = a.out != nullptr;
    LisLaunch p;
    p.ntiles = (a.Lq + kRowsPerBlock - 1) / kRowsPerBlock;
    const int nc = (a.Lk + 31) / 32;
    // V^T columns padded to a power of two, at least 32 (two MFMA tiles).
    int dt = 2;
    while (fused && 16 * dt < a.d) dt <<= 1;
    p.dpad = 16 * dt;
    p.ncg = dt;
    const int max_keys = vt_stage_keys(p.dpad);
    p.kb = std::max(32, std::min(nc * 32, max_keys));
    p.ld = p.kb + 8;
    p.vec_ok = fused && (a.d % 16 == 0) && ((reinterpret_cast<uintptr_t>(a.v) & 15) == 0);
    p.vt_bytes = fused ? p.dpad * p.ld * (int)sizeof(uint16_t) : 0;
    p.out_vec = fused && (a.d % 4 == 0) && ((reinterpret_cast<uintptr_t>(a.out) & 15) == 0);
    // LDS of the row-wise output stores: one 16 x (dpad + 4) int32 block per wavefront
    const size_t out_lds = p.out_vec ? (size_t)4 * 16 * (p.dpad + 4) * sizeof(int32_t) : 0;
    p.n_logits = a.G * (int64_t)a.Lq * a.Lk;
    p.n_bias = a.bias ? (int64_t)a.Hb * a.Lq * a.Lk : 0;
    p.tab_bytes = 0;
    p.codes_ldw = 0;
    const int64_t blocks = a.G * (int64_t)p.ntiles;
    const dim3 grid((unsigned)blocks);
    const bool fp = a.k.fp_ok != 0;
    // Unit kernel: rows of up to 224 keys on the float path, V^T in one stage,
    // and enough units to give every SIMD two busy wavefronts.
    const int tiles16 = (a.Lq + 15) / 16;
    const bool unit_ok = nc <= kUnitMaxNC && fp && (!fused || (a.codes == nullptr && dt <= 4)) &&
                         a.G <= 0x7FFFFFFF && a.G * std::min(4, tiles16) >= 2048;
    if (unit_ok) {
        LisLaunch u = p;
        u.ntiles = tiles16;
        u.kb = nc * 32;
        u.ld = u.kb + 8;
        u.vt_bytes = fused ? u.dpad * u.ld * (int)sizeof(uint16_t) : 0;
        const int wpu = unit_waves(nc, tiles16);
        size_t lds = (size_t)u.vt_bytes + out_lds / 4 * wpu;
        // codes only, dense rows: each wavefront gathers its tile's code rows
        // in LDS and writes them as one span
        const int row_bytes = a.k.top > 15 ? a.Lk : (a.Lk + 1) / 2;
        if (!fused && a.ld_codes == row_bytes) {
            u.codes_ldw = (16 * row_bytes + 8 + 15) / 16 * 16;
            lds += (size_t)wpu * u.codes_ldw;
        }
        const bool half = a.Lk - 32 * (nc - 1) <= 16;
        return launch_lis_unit(nc, fused, dt, half, wpu, a, u, lds, stream);
    }
    // Long-row kernel: fused rows of 10 to 20 chunks on the float path, d <= 64,
    // no codes output, when its I-Exp table (u_max + 1 entries, byte offsets in
    // 16 bits) and V^T fit the LDS of one workgroup.
    const bool long_ok = fused && fp && a.codes == nullptr && dt <= 4 && nc >= kLongMinNC &&
                         nc <= kLongMaxNC && a.G <= 0x7FFFFFFF && a.k.u_max <= 16383 &&
                         (int64_t)a.Lq * a.Lk * 4 < ((int64_t)1 << 31);
    if (long_ok) {
        LisLaunch l = p;
        l.ntiles = tiles16;
        l.kb = nc * 32;
        l.ld = l.kb + 8;
        l.vt_bytes = l.dpad * l.ld * (int)sizeof(uint16_t);
        l.tab_bytes = (int)((((int64_t)a.k.u_max + 1) * 4 + 15) / 16 * 16);
        const size_t lds = (size_t)l.tab_bytes + (size_t)l.vt_bytes;
        if (lds <= kMaxLdsBytes) {
            const bool half = a.Lk - 32 * (nc - 1) <= 16;
            return nc <= 14 ? launch_lis_long_lo(nc, dt, half, a, l, lds, stream)
                            : launch_lis_long_hi(nc, dt, half, a, l, lds, stream);
        }
    }
    // Tile kernels: codes only for rows of up to 640 keys, the fused product
    // (without a codes output, d <= 64) for rows of up to 288 keys.
    const bool regs = fused ? (nc <= kRegsFusedMaxNC && a.codes == nullptr && dt <= 4) : nc <= 20;
    if (regs) {
        const size_t lds = (size_t)p.vt_bytes + out_lds;
        return nc <= 10 ? launch_lis_regs_lo(nc, fused, dt, fp, a, p, grid, lds, stream)
                        : launch_lis_regs_hi(nc, fused, dt, fp, a, p, grid, lds, stream);
    }
    const size_t lds = fused ? (size_t)p.vt_bytes : 0;
    if (fp)
        launch_stream<true>(fused, dt, grid, lds, stream, a, p);
    else
        launch_stream<false>(fused, dt, grid, lds, stream, a, p);
    return hipGetLastError();
}

hipError_t launch_attn_v_shift(const AvArgs& a, hipStream_t stream) {
    using lis::kBlock;
    const hipError_t mf = launch_attn_v_mfma(a, stream);
    if (mf != hipErrorNotSupported) return mf;
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
    launch_kernel(lis::attn_v_shift_kernel, dim3((unsigned)blocks), dim3(kBlock), lds, stream, a,
                       tpr, rows, ntiles, kb);
    return hipGetLastError();
}

hipError_t launch_attn_v_shift_wide(const AvWideArgs& a, hipStream_t stream) {
    using lis::kBlock;
    const hipError_t mf = launch_attn_v_wide_mfma(a, stream);
    if (mf != hipErrorNotSupported) return mf;
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
    launch_kernel(lis::attn_v_shift_wide_kernel, dim3((unsigned)blocks), dim3(kBlock), lds, stream,
                  a, tpr, rows, ntiles, kb);
    return hipGetLastError();
}

}  // namespace fqvit
