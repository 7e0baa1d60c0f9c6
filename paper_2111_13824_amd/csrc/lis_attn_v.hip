// Standalone BitShift Attn x V (Sec. 3.3 and the zero-point form of
// Supplement A.2) on the int8 matrix cores of gfx950:
//   out[g, i, c] = sum_j (v[g, j, c] - zp_V) 2^(N - code[g, i, j]),  N = 2^b - 1,
// exact in int32 (modulo 2^32) for any codes 0..N (a code above N, which
// Log-Int-Softmax never writes, gives an unspecified result).
//
// P = 2^s with s = N - code in [0, 15] is split into 7-bit exponent ranges,
// P = sum_k 2^(7 k) P_k with P_k = 2^(s - 7 k) for 7 k <= s < 7 k + 7 (else
// 0), so every P_k is at most 64 and fits int8 beside V itself.  Then
//   out = sum_k 2^(7 k) (V^T P_k^T) - zp_V sum_j P_j,
// where each product V^T P_k^T is one v_mfma_i32_16x16x64_i8 per 64 keys and
// 16 x 16 outputs, its int32 sums bounded by 128 * 64 * 4096 = 2^25 (exact),
// and the recombination is done modulo 2^32, as the product's definition
// asks.  b <= 2 needs one range (s <= 3), b = 3 two (s <= 7), b = 4 three.
//
// One workgroup of four wavefronts per attention unit: V^T of the unit is
// staged in LDS as int8 (keys padded to a multiple of 64 with zeros, in the
// byte order of the code expansion below); each wavefront walks the unit's
// 16-row tiles.  Lane (r, kq) takes query row i0 + r and keys
// 64 ks + 16 kq .. + 15 of each 64-key step: their eight code bytes (nibble
// pairs) come straight from memory as three aligned dwords and a funnel shift,
// the nibbles are spread into bytes (keys 0,2,4,6 | 1,3,5,7 | 8,10,.. |
// 9,11,..), and each P_k byte is a table lookup (two byte permutes and a
// select on the code's bit 3).  The B operand of the MFMA is P_k^T (keys x
// rows), the A operand V^T (columns x keys), so the output lane (r, kq) holds
// columns 16 ct + 4 kq .. + 3 of row i0 + r: one 16-byte store.
#include "fqvit_launch.h"
#include "lis_device.h"

namespace fqvit {
namespace lis {
namespace {

typedef int32_t av_i32x4 __attribute__((ext_vector_type(4)));

// key offset (0..15) of byte p of a lane's 16 expanded code bytes
__device__ __forceinline__ int av_key_of_byte(int p) {
    return (p & 8) | ((p & 3) << 1) | ((p >> 2) & 1);
}

// V^T of the unit in LDS.  Fast form (m.vec_v: d % 16 == 0, 16-byte aligned
// V): item = (key quad, 16-column group); the four keys of byte positions
// 4 q .. 4 q + 3 are read as four 16-byte rows and transposed in registers,
// so that each of the 16 columns gets one dword store.  Otherwise one byte
// at a time.
template <int DT>
__device__ __forceinline__ void av_stage_vt(uint8_t* vt, const int8_t* vg, const AvArgs& a,
                                            const AvMfma& m) {
    const int Lk = a.Lk;
    const int d = a.d;
    const int nq = m.kp / 4;
    if (m.vec_v) {
        const int ncg = d / 16;
        for (int idx = threadIdx.x; idx < nq * DT; idx += 256) {
            const int cg = idx / nq;
            const int q = idx - cg * nq;
            uint32_t x[4][4];
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const int key = 16 * (q >> 2) + av_key_of_byte(4 * (q & 3) + t);
                av_i32x4 row = {0, 0, 0, 0};
                if (key < Lk && cg < ncg)
                    row = *reinterpret_cast<const av_i32x4*>(vg + (int64_t)key * d + 16 * cg);
#pragma unroll
                for (int u = 0; u < 4; ++u) x[t][u] = (uint32_t)row[u];
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                // columns 16 cg + 4 u .. + 3: a 4 x 4 byte transpose
                const uint32_t lo01 = __builtin_amdgcn_perm(x[1][u], x[0][u], 0x05010400u);
                const uint32_t hi01 = __builtin_amdgcn_perm(x[1][u], x[0][u], 0x07030602u);
                const uint32_t lo23 = __builtin_amdgcn_perm(x[3][u], x[2][u], 0x05010400u);
                const uint32_t hi23 = __builtin_amdgcn_perm(x[3][u], x[2][u], 0x07030602u);
                const int c = 16 * cg + 4 * u;
                *reinterpret_cast<uint32_t*>(vt + (c + 0) * m.ldv + 4 * q) = __builtin_amdgcn_perm(lo23, lo01, 0x05040100u);
                *reinterpret_cast<uint32_t*>(vt + (c + 1) * m.ldv + 4 * q) = __builtin_amdgcn_perm(lo23, lo01, 0x07060302u);
                *reinterpret_cast<uint32_t*>(vt + (c + 2) * m.ldv + 4 * q) = __builtin_amdgcn_perm(hi23, hi01, 0x05040100u);
                *reinterpret_cast<uint32_t*>(vt + (c + 3) * m.ldv + 4 * q) = __builtin_amdgcn_perm(hi23, hi01, 0x07060302u);
            }
        }
    } else {
        for (int idx = threadIdx.x; idx < 16 * DT * nq; idx += 256) {
            const int q = idx / (16 * DT);
            const int c = idx - q * (16 * DT);
            uint32_t w = 0;
            if (c < d) {
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    const int key = 16 * (q >> 2) + av_key_of_byte(4 * (q & 3) + t);
                    if (key < Lk) w |= (uint32_t)(uint8_t)vg[(int64_t)key * d + c] << (8 * t);
                }
            }
            *reinterpret_cast<uint32_t*>(vt + c * m.ldv + 4 * q) = w;
        }
    }
}

// Three aligned dwords holding the eight code bytes of lane (r, kq) in step ks
// of its row at byte offset rowoff (relative to the aligned unit base);
// rowoff < 0: nothing (past the buffer, no memory access).
__device__ __forceinline__ void av_load_codes(uint32_t (&w)[3], __amdgpu_buffer_rsrc_t cr,
                                              int rowoff, int ks, int kq) {
    const int o = rowoff < 0 ? INT_MIN : (rowoff + 32 * ks + 8 * kq) & ~3;
#pragma unroll
    for (int t = 0; t < 3; ++t)
        w[t] = __builtin_amdgcn_raw_buffer_load_b32(cr, rowoff < 0 ? INT_MIN : o + 4 * t, 0, 0);
}

constexpr int kAvWin = 4;   // 64-key steps whose codes are in flight per wavefront

// Ranges of P = 2^(N - code) for b bits: NS ranges of 7 exponents; range k
// holds codes N - 7 k - 6 .. N - 7 k, so it needs the table half of codes 0..7
// (AV_LO) and / or 8..15 (AV_HI).
template <int B>
struct AvRanges {
    static constexpr int N = (1 << B) - 1;
    static constexpr int NS = N / 7 + 1;
    static constexpr bool lo(int k) { return (N - 7 * k - 6 > 0 ? N - 7 * k - 6 : 0) <= 7; }
    static constexpr bool hi(int k) { return N - 7 * k >= 8; }
};

// ZS: the zero point is not 0, so sum_j P_j is needed.
template <int DT, int B, bool ZS>
__global__ __launch_bounds__(256) void attn_v_mfma_kernel(AvArgs a, AvMfma m) {
    using R = AvRanges<B>;
    constexpr int NS = R::NS;
    extern __shared__ __attribute__((aligned(16))) uint8_t vt[];   // [16 DT][ldv] int8
    const int64_t g = xcd_remap(blockIdx.x, a.G);
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int r = lane & 15;
    const int kq = lane >> 4;
    const int Lk = a.Lk;
    const int d = a.d;
    const int nks = m.nks;

    // the unit's codes as dwords from an aligned base (reads past the unit's
    // last code byte return 0: they only ever hold keys past Lk)
    const uint64_t ubase = (uint64_t)(a.codes + g * a.Lq * (int64_t)a.ld_codes);
    const int mis = (int)(ubase & 3);
    const __amdgpu_buffer_rsrc_t cr = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(ubase - (uint64_t)mis), (short)0, (m.unit_bytes + mis + 3) & ~3, 0x00020000);

    // The wavefront's steps: tiles wave, wave + 4, ..., each in nks steps of
    // 64 keys.  The codes of the next kAvWin steps are in flight: (pt, pks)
    // is the step whose codes are requested next.  The first window is
    // requested before V^T is staged.
    const int my_tiles = m.ntiles > wave ? (m.ntiles - wave + 3) / 4 : 0;
    const int nsteps = my_tiles * nks;
    auto row_of = [&](int t) {
        return t < m.ntiles ? min(16 * t + r, a.Lq - 1) * a.ld_codes + mis : -1;
    };
    int pt = wave, pks = 0;
    int prow = row_of(pt);
    uint32_t cb[kAvWin][3];
#pragma unroll
    for (int u = 0; u < kAvWin; ++u) {
        av_load_codes(cb[u], cr, prow, pks, kq);
        if (++pks == nks) {
            pks = 0;
            pt += 4;
            prow = row_of(pt);
        }
    }

    av_stage_vt<DT>(vt, a.v + g * (int64_t)Lk * d, a, m);
    __syncthreads();

    const uint32_t zpu = (uint32_t)a.zp_v;
    // sum_j P_j (with a zero point only) must leave out the keys past Lk in
    // the last step (their V^T is zero, so the products need no mask)
    uint32_t keep_last[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        uint32_t km = 0;
#pragma unroll
        for (int t = 0; t < 4; ++t)
            km |= (64 * (nks - 1) + 16 * kq + av_key_of_byte(4 * q + t) < Lk ? 0xFFu : 0u) << (8 * t);
        keep_last[q] = km;
    }
    av_i32x4 acc[DT][NS];
    uint32_t psum[NS];
    int ks = 0, tile = wave;
    int rowoff = row_of(tile);
    for (int s0 = 0; s0 < nsteps; s0 += kAvWin) {
#pragma unroll
        for (int u = 0; u < kAvWin; ++u) {
            const int s = s0 + u;
            if (s >= nsteps) break;
            if (ks == 0) {
#pragma unroll
                for (int ct = 0; ct < DT; ++ct)
#pragma unroll
                    for (int k = 0; k < NS; ++k) acc[ct][k] = av_i32x4{0, 0, 0, 0};
#pragma unroll
                for (int k = 0; k < NS; ++k) psum[k] = 0;
            }
            const int sh = (rowoff + 32 * ks + 8 * kq) & 3;
            const uint32_t lo = __builtin_amdgcn_alignbyte(cb[u][1], cb[u][0], sh);
            const uint32_t hi = __builtin_amdgcn_alignbyte(cb[u][2], cb[u][1], sh);
            av_load_codes(cb[u], cr, prow, pks, kq);
            if (++pks == nks) {
                pks = 0;
                pt += 4;
                prow = row_of(pt);
            }
            const uint32_t cw[4] = {lo & 0x0F0F0F0Fu, (lo >> 4) & 0x0F0F0F0Fu, hi & 0x0F0F0F0Fu,
                                    (hi >> 4) & 0x0F0F0F0Fu};
            const bool last = ks == nks - 1;
            av_i32x4 Bop[NS];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const uint32_t sel = cw[q] & 0x07070707u;
                // 0xFF in the bytes of codes >= 8 (b = 4 only: for b <= 3 a
                // code above 7 is not a valid code)
                uint32_t hib = 0;
                if (B == 4)   // byte select 0 -> 0x00, 1 -> 0xFF
                    hib = __builtin_amdgcn_perm(0u, 0x0000FF00u, (cw[q] >> 3) & 0x01010101u);
#pragma unroll
                for (int k = 0; k < NS; ++k) {
                    uint32_t pb;
                    if (R::lo(k) && R::hi(k)) {
                        const uint32_t plo = __builtin_amdgcn_perm(m.lut[k][1], m.lut[k][0], sel);
                        const uint32_t phi = __builtin_amdgcn_perm(m.lut[k][3], m.lut[k][2], sel);
                        pb = (phi & hib) | (plo & ~hib);
                    } else if (R::hi(k)) {
                        pb = __builtin_amdgcn_perm(m.lut[k][3], m.lut[k][2], sel) & hib;
                    } else if (B == 4) {
                        pb = __builtin_amdgcn_perm(m.lut[k][1], m.lut[k][0], sel) & ~hib;
                    } else {
                        pb = __builtin_amdgcn_perm(m.lut[k][1], m.lut[k][0], sel);
                    }
                    Bop[k][q] = (int32_t)pb;
                    if (ZS)
                        psum[k] = __builtin_amdgcn_udot4(last ? pb & keep_last[q] : pb, 0x01010101u,
                                                         psum[k], false);
                }
            }
#pragma unroll
            for (int ct = 0; ct < DT; ++ct) {
                const av_i32x4 A =
                    *reinterpret_cast<const av_i32x4*>(vt + (16 * ct + r) * m.ldv + 64 * ks + 16 * kq);
#pragma unroll
                for (int k = 0; k < NS; ++k)
                    acc[ct][k] = __builtin_amdgcn_mfma_i32_16x16x64_i8(A, Bop[k], acc[ct][k], 0, 0, 0);
            }
            if (++ks == nks) {
                // the tile's output: sum_j P_j of row i0 + r over the four
                // key groups, then the recombined ranges less zp_V sum_j P_j
                uint32_t zterm = 0;
                if (ZS) {
                    uint32_t pt = 0;
#pragma unroll
                    for (int k = 0; k < NS; ++k) pt += psum[k] << (7 * k);
                    pt += (uint32_t)__shfl_xor((int)pt, 16, 64);
                    pt += (uint32_t)__shfl_xor((int)pt, 32, 64);
                    zterm = zpu * pt;
                }
                const int row = 16 * tile + r;
                if (row < a.Lq) {
                    int32_t* orow = a.out + (g * a.Lq + row) * (int64_t)d;
#pragma unroll
                    for (int ct = 0; ct < DT; ++ct) {
                        uint32_t res[4];
#pragma unroll
                        for (int t = 0; t < 4; ++t) {
                            uint32_t v = (uint32_t)acc[ct][0][t];
                            if (NS > 1) v += (uint32_t)acc[ct][NS > 1 ? 1 : 0][t] << 7;
                            if (NS > 2) v += (uint32_t)acc[ct][NS > 2 ? 2 : 0][t] << 14;
                            res[t] = v - zterm;
                        }
                        const int c0 = 16 * ct + 4 * kq;
                        if (m.vec_out && c0 + 3 < d) {
                            *reinterpret_cast<av_i32x4*>(orow + c0) =
                                av_i32x4{(int32_t)res[0], (int32_t)res[1], (int32_t)res[2], (int32_t)res[3]};
                        } else {
#pragma unroll
                            for (int t = 0; t < 4; ++t)
                                if (c0 + t < d) orow[c0 + t] = (int32_t)res[t];
                        }
                    }
                }
                ks = 0;
                tile += 4;
                rowoff = row_of(tile);
            }
        }
    }
}

template <int DT, bool ZS>
hipError_t launch_dt(int bits, const AvArgs& a, const AvMfma& m, size_t lds, hipStream_t s) {
    const dim3 grid((unsigned)a.G), block(256);
    switch (bits) {
        case 1: launch_kernel(attn_v_mfma_kernel<DT, 1, ZS>, grid, block, lds, s, a, m); break;
        case 2: launch_kernel(attn_v_mfma_kernel<DT, 2, ZS>, grid, block, lds, s, a, m); break;
        case 3: launch_kernel(attn_v_mfma_kernel<DT, 3, ZS>, grid, block, lds, s, a, m); break;
        default: launch_kernel(attn_v_mfma_kernel<DT, 4, ZS>, grid, block, lds, s, a, m); break;
    }
    return hipGetLastError();
}

template <int DT>
hipError_t launch_dtz(int bits, const AvArgs& a, const AvMfma& m, size_t lds, hipStream_t s) {
    return a.zp_v != 0 ? launch_dt<DT, true>(bits, a, m, lds, s) : launch_dt<DT, false>(bits, a, m, lds, s);
}

}  // namespace
}  // namespace lis

hipError_t launch_attn_v_mfma(const AvArgs& a, hipStream_t stream) {
    using namespace lis;
    AvMfma m;
    m.kp = (a.Lk + 63) / 64 * 64;
    m.nks = m.kp / 64;
    m.ldv = m.kp + 16;
    m.ntiles = (a.Lq + 15) / 16;
    m.vec_out = (a.d % 4 == 0) && ((reinterpret_cast<uintptr_t>(a.out) & 15) == 0);
    m.vec_v = (a.d % 16 == 0) && ((reinterpret_cast<uintptr_t>(a.v) & 15) == 0);
    // the unit's code bytes: rows 0 .. Lq - 1 at stride ld_codes, ceil(Lk/2) each
    const int64_t ub = (int64_t)(a.Lq - 1) * a.ld_codes + (a.Lk + 1) / 2;
    int dt = 1;
    while (16 * dt < a.d) dt <<= 1;
    const size_t lds = (size_t)16 * dt * m.ldv;
    if (dt > 4 || a.Lk > kAvMfmaMaxLk || ub + 6 > 0x7FFFFFFF || a.G > 0x7FFFFFFF)
        return hipErrorNotSupported;
    m.unit_bytes = (int)ub;
    // P_k byte tables: code c -> 2^(s - 7 k) for 7 k <= s < 7 k + 7, s = top - c
    const int bits = a.top == 15 ? 4 : a.top == 7 ? 3 : a.top == 3 ? 2 : 1;
    for (int k = 0; k < 3; ++k) {
        for (int w = 0; w < 4; ++w) m.lut[k][w] = 0;
        for (int c = 0; c < 16; ++c) {
            const int s = a.top - c;
            const uint32_t byte = (s >= 7 * k && s < 7 * k + 7) ? (1u << (s - 7 * k)) : 0u;
            m.lut[k][c >> 2] |= byte << (8 * (c & 3));
        }
    }
    switch (dt) {
        case 1: return launch_dtz<1>(bits, a, m, lds, stream);
        case 2: return launch_dtz<2>(bits, a, m, lds, stream);
        default: return launch_dtz<4>(bits, a, m, lds, stream);
    }
}

}  // namespace fqvit
