// BitShift Attn x V (Sec. 3.3 and the zero-point form of Supplement A.2) on the
// int8 matrix cores of gfx950, for the standalone products:
//   narrow: out[g, i, c] = sum_j (v[g, j, c] - zp_V) 2^(N - code[g, i, j]) in
//           int32 (modulo 2^32), N = 2^b - 1, b <= 4, nibble codes; a code
//           above N (never written by Log-Int-Softmax) gives an unspecified
//           result;
//   wide:   out[g, i, c] = sum_j floor((v[g, j, c] - zp_V) 2^(W - code[g, i, j]))
//           in int64 (modulo 2^64), W = min(2^b - 1, 44), nibble codes for
//           b <= 4 and byte codes above.
//
// With s = W - code (W = N for the narrow product) and s >= 0, P = 2^s is
// split into ranges of seven exponents, P = sum_k 2^(7 k) P_k with
// P_k = 2^(s - 7 k) on 7 k <= s < 7 k + 7 and 0 elsewhere, so every P_k is at
// most 64 and fits int8 beside V itself.  Then
//   out = sum_k 2^(7 k) (V^T P_k^T) - zp_V sum_j P_j,
// each V^T P_k^T one v_mfma_i32_16x16x64_i8 per 64 keys and 16 x 16 outputs,
// its int32 sums bounded by 128 * 64 * 4096 = 2^25 (exact).  The ranges are
// recombined modulo 2^32 (narrow) or 2^64 (wide), as the products are
// defined.  Ranges: b <= 2 one, b = 3 two, b = 4 three, b = 5 five (W = 31),
// b >= 6 seven (W = 44).  A code above W (wide product only, never made by
// Log-Int-Softmax) contributes the floor of a right shift, which the ranges
// cannot express: a unit holding one is computed again afterwards, exactly,
// on the vector ALUs (from the V^T staged for it).
//
// One workgroup of four wavefronts per attention unit: V^T of the unit is
// staged in LDS as int8 (keys padded to a multiple of 64 with zeros); each
// wavefront walks the unit's 16-row tiles.  Lane (r, kq) takes query row
// i0 + r and keys 64 ks + 16 kq .. + 15 of each 64-key step, its code bytes
// straight from memory as aligned dwords and funnel shifts:
//   * nibble codes: eight bytes, the nibbles spread into bytes (keys
//     0,2,4,6 | 1,3,5,7 | 8,10,.. | 9,11,..; V^T is staged in the same key
//     order), each P_k byte a table lookup (one or two byte permutes over
//     8-entry tables chosen at compile time, and a select on the code's bit 3);
//   * byte codes: sixteen bytes in key order; per key the 64-bit value
//     2^(8 k + e) (s = 7 k + e) holds its P_k in byte k, and a 4 x 8 byte
//     transpose of four keys gives the range dwords.
// The B operand of the MFMA is P_k^T (keys x rows), the A operand V^T
// (columns x keys), so the output lane (r, kq) holds columns 16 ct + 4 kq .. + 3
// of row i0 + r.  The codes of the next four (nibble codes) or two (byte
// codes) steps are in flight per wavefront across tile boundaries, and the
// kernel is held to two wavefronts per SIMD (at most 256 registers).
#include "fqvit_launch.h"
#include "lis_device.h"

namespace fqvit {
namespace lis {
namespace {

typedef int32_t av_i32x4 __attribute__((ext_vector_type(4)));

// Arguments shared by both products.
struct AvK {
    const uint8_t* codes;
    int32_t ld_codes;
    const int8_t* v;
    int32_t zp_v;
    int64_t G;
    int32_t Lq, Lk, d;
    int32_t W;          // output exponent (N for the narrow product)
    void* out;          // int32 (narrow) or int64 (wide) [G, Lq, d]
};

// key offset (0..15) of byte p of a lane's 16 expanded nibble-code bytes, and
// the byte position of key offset u
__device__ __forceinline__ int av_key_of_byte(int p) {
    return (p & 8) | ((p & 3) << 1) | ((p >> 2) & 1);
}
__device__ __forceinline__ int av_byte_of_key(int u) {
    return (u & 8) + ((u & 1) << 2) + ((u & 7) >> 1);
}

// y[b] = the bytes {x0.b, x1.b, x2.b, x3.b}: a 4 x 4 byte transpose
__device__ __forceinline__ void av_transpose4(uint32_t (&y)[4], uint32_t x0, uint32_t x1,
                                              uint32_t x2, uint32_t x3) {
    const uint32_t lo01 = __builtin_amdgcn_perm(x1, x0, 0x05010400u);
    const uint32_t hi01 = __builtin_amdgcn_perm(x1, x0, 0x07030602u);
    const uint32_t lo23 = __builtin_amdgcn_perm(x3, x2, 0x05010400u);
    const uint32_t hi23 = __builtin_amdgcn_perm(x3, x2, 0x07030602u);
    y[0] = __builtin_amdgcn_perm(lo23, lo01, 0x05040100u);
    y[1] = __builtin_amdgcn_perm(lo23, lo01, 0x07060302u);
    y[2] = __builtin_amdgcn_perm(hi23, hi01, 0x05040100u);
    y[3] = __builtin_amdgcn_perm(hi23, hi01, 0x07060302u);
}

// V^T of the unit in LDS, the keys of each 16-key group at the byte positions
// of the code expansion (PI: nibble order, else key order).  Fast form
// (m.vec_v: d % 16 == 0, 16-byte aligned V): item = (key quad, 16-column
// group), four 16-byte rows transposed in registers, one dword store per
// column.  Otherwise one byte at a time.
template <int DT, bool PI>
__device__ __forceinline__ void av_stage_vt(uint8_t* vt, const int8_t* vg, const AvK& a,
                                            const AvMfma& m) {
    const int Lk = a.Lk;
    const int d = a.d;
    const int nq = m.kp / 4;
    auto key_at = [](int q, int t) {
        const int p = 4 * (q & 3) + t;
        return 16 * (q >> 2) + (PI ? av_key_of_byte(p) : p);
    };
    if (m.vec_v) {
        const int ncg = d / 16;
        for (int idx = threadIdx.x; idx < nq * DT; idx += 256) {
            const int cg = idx / nq;
            const int q = idx - cg * nq;
            uint32_t x[4][4];
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const int key = key_at(q, t);
                av_i32x4 row = {0, 0, 0, 0};
                if (key < Lk && cg < ncg)
                    row = *reinterpret_cast<const av_i32x4*>(vg + (int64_t)key * d + 16 * cg);
#pragma unroll
                for (int u = 0; u < 4; ++u) x[t][u] = (uint32_t)row[u];
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                uint32_t y[4];
                av_transpose4(y, x[0][u], x[1][u], x[2][u], x[3][u]);
                const int c = 16 * cg + 4 * u;
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    *reinterpret_cast<uint32_t*>(vt + (c + e) * m.ldv + 4 * q) = y[e];
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
                    const int key = key_at(q, t);
                    if (key < Lk) w |= (uint32_t)(uint8_t)vg[(int64_t)key * d + c] << (8 * t);
                }
            }
            *reinterpret_cast<uint32_t*>(vt + c * m.ldv + 4 * q) = w;
        }
    }
}

// The aligned dwords holding the code bytes of lane (r, kq) in step ks of its
// row at byte offset rowoff (relative to the aligned unit base); rowoff < 0:
// nothing (past the buffer, no memory access).  BYTES: 16 bytes per lane and
// step (five dwords), else 8 (three dwords).
template <bool BYTES>
__device__ __forceinline__ void av_load_codes(uint32_t (&w)[BYTES ? 5 : 3],
                                              __amdgpu_buffer_rsrc_t cr, int rowoff, int ks,
                                              int kq) {
    constexpr int NW = BYTES ? 5 : 3;
    const int o = BYTES ? rowoff + 64 * ks + 16 * kq : rowoff + 32 * ks + 8 * kq;
#pragma unroll
    for (int t = 0; t < NW; ++t)
        w[t] = __builtin_amdgcn_raw_buffer_load_b32(cr, rowoff < 0 ? INT_MIN : (o & ~3) + 4 * t, 0, 0);
}

// Ranges of P = 2^(N - code) for b-bit nibble codes: NS ranges of 7 exponents;
// range k holds codes N - 7 k - 6 .. N - 7 k, so it needs the table half of
// codes 0..7 (lo) and / or 8..15 (hi).
template <int B>
struct AvRanges {
    static constexpr int N = (1 << B) - 1;
    static constexpr int NS = N / 7 + 1;
    static constexpr bool lo(int k) { return (N - 7 * k - 6 > 0 ? N - 7 * k - 6 : 0) <= 7; }
    static constexpr bool hi(int k) { return N - 7 * k >= 8; }
};

// 64-key steps whose codes are in flight per wavefront (byte codes: fewer,
// so that the seven range accumulators leave room for two wavefronts per SIMD)
template <bool BYTES>
constexpr int av_win() { return BYTES ? 2 : 4; }

// CB: code width (1..4 bits: nibbles; 5: bytes, W = 31; 8: bytes, W = 44);
// ZS: the zero point is not 0 (sum_j P_j needed); WIDE: int64 output, with
// the floor of codes above W.
template <int DT, int CB, bool ZS, bool WIDE>
__global__ __launch_bounds__(256, 2) void attn_v_mfma_kernel(AvK a, AvMfma m) {
    constexpr bool BYTES = CB >= 5;
    constexpr int kAvWin = av_win<BYTES>();
    using R = AvRanges<BYTES ? 1 : CB>;
    constexpr int NS = BYTES ? (CB == 5 ? 5 : 7) : R::NS;
    constexpr int NW = BYTES ? 5 : 3;
    extern __shared__ __attribute__((aligned(16))) uint8_t vt[];   // [16 DT][ldv] int8
    __shared__ int s_floor;
    const int64_t g = xcd_remap(blockIdx.x, a.G);
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int r = lane & 15;
    const int kq = lane >> 4;
    const int Lk = a.Lk;
    const int d = a.d;
    const int nks = m.nks;
    if (threadIdx.x == 0) s_floor = 0;

    // the unit's codes as dwords from an aligned base (reads past the unit's
    // last code byte return 0: they only ever hold keys past Lk)
    const uint64_t ubase = (uint64_t)(a.codes + g * a.Lq * (int64_t)a.ld_codes);
    const int mis = (int)(ubase & 3);
    const __amdgpu_buffer_rsrc_t cr = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(ubase - (uint64_t)mis), (short)0, (m.unit_bytes + mis + 3) & ~3, 0x00020000);

    // The wavefront's steps: tiles wave, wave + 4, ..., each in nks steps of
    // 64 keys; (pt, pks) is the step whose codes are requested next.  The first
    // window is requested before V^T is staged.
    const int my_tiles = m.ntiles > wave ? (m.ntiles - wave + 3) / 4 : 0;
    const int nsteps = my_tiles * nks;
    auto row_of = [&](int t) {
        return t < m.ntiles ? min(16 * t + r, a.Lq - 1) * a.ld_codes + mis : -1;
    };
    int pt = wave, pks = 0;
    int prow = row_of(pt);
    uint32_t cb[kAvWin][NW];
#pragma unroll
    for (int u = 0; u < kAvWin; ++u) {
        av_load_codes<BYTES>(cb[u], cr, prow, pks, kq);
        if (++pks == nks) {
            pks = 0;
            pt += 4;
            prow = row_of(pt);
        }
    }

    av_stage_vt<DT, !BYTES>(vt, a.v + g * (int64_t)Lk * d, a, m);
    __syncthreads();

    // keys past Lk in the last step: left out of sum_j P_j (their V^T is zero,
    // so the products need no mask) and of the search for codes above W
    uint32_t keep_last[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        uint32_t km = 0;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const int p = 4 * q + t;
            const int key = 64 * (nks - 1) + 16 * kq + (BYTES ? p : av_key_of_byte(p));
            km |= (key < Lk ? 0xFFu : 0u) << (8 * t);
        }
        keep_last[q] = km;
    }
    // nibble codes above W (b <= 3; the wide product only)
    const uint32_t over_mask = (uint32_t)(~a.W & 15) * 0x01010101u;
    bool floor_seen = false;

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
            const int sh = (BYTES ? rowoff + 64 * ks + 16 * kq : rowoff + 32 * ks + 8 * kq) & 3;
            uint32_t cw[4];
            if constexpr (BYTES) {
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    cw[q] = __builtin_amdgcn_alignbyte(cb[u][q + 1], cb[u][q], sh);
            } else {
                const uint32_t lo = __builtin_amdgcn_alignbyte(cb[u][1], cb[u][0], sh);
                const uint32_t hi = __builtin_amdgcn_alignbyte(cb[u][2], cb[u][1], sh);
                cw[0] = lo & 0x0F0F0F0Fu;
                cw[1] = (lo >> 4) & 0x0F0F0F0Fu;
                cw[2] = hi & 0x0F0F0F0Fu;
                cw[3] = (hi >> 4) & 0x0F0F0F0Fu;
            }
            av_load_codes<BYTES>(cb[u], cr, prow, pks, kq);
            if (++pks == nks) {
                pks = 0;
                pt += 4;
                prow = row_of(pt);
            }
            const bool last = ks == nks - 1;
            av_i32x4 Bop[NS];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const uint32_t kmask = last ? keep_last[q] : ~0u;
                uint32_t pb[NS];
                if constexpr (BYTES) {
                    // per key: s = W - code; 2^(8 k + e) with s = 7 k + e holds
                    // P_k in byte k (floor(37 s / 256) = floor(s / 7) for s <= 44)
                    uint32_t xl[4], xh[4];
#pragma unroll
                    for (int t = 0; t < 4; ++t) {
                        const int c = (int)((cw[q] >> (8 * t)) & 0xFFu);
                        const int sv = a.W - c;
                        if (WIDE) floor_seen |= sv < 0 && ((kmask >> (8 * t)) & 1u);
                        const int kk = (sv * 37) >> 8;
                        const uint64_t x = sv >= 0 ? (uint64_t)1 << (sv + kk) : 0ull;
                        xl[t] = (uint32_t)x;
                        xh[t] = (uint32_t)(x >> 32);
                    }
                    uint32_t y[4];
                    av_transpose4(y, xl[0], xl[1], xl[2], xl[3]);
#pragma unroll
                    for (int k = 0; k < 4; ++k) pb[k] = y[k];
                    av_transpose4(y, xh[0], xh[1], xh[2], xh[3]);
#pragma unroll
                    for (int k = 4; k < NS; ++k) pb[k] = y[k - 4];
                } else {
                    if (WIDE && R::N < 15) floor_seen |= (cw[q] & over_mask & kmask) != 0;
                    const uint32_t sel = cw[q] & 0x07070707u;
                    // 0xFF in the bytes of codes >= 8 (b = 4 only: for b <= 3
                    // a code above 7 is above N)
                    uint32_t hib = 0;
                    if (CB == 4)   // byte select 0 -> 0x00, 1 -> 0xFF
                        hib = __builtin_amdgcn_perm(0u, 0x0000FF00u, (cw[q] >> 3) & 0x01010101u);
#pragma unroll
                    for (int k = 0; k < NS; ++k) {
                        if (R::lo(k) && R::hi(k)) {
                            const uint32_t plo = __builtin_amdgcn_perm(m.lut[k][1], m.lut[k][0], sel);
                            const uint32_t phi = __builtin_amdgcn_perm(m.lut[k][3], m.lut[k][2], sel);
                            pb[k] = (phi & hib) | (plo & ~hib);
                        } else if (R::hi(k)) {
                            pb[k] = __builtin_amdgcn_perm(m.lut[k][3], m.lut[k][2], sel) & hib;
                        } else if (CB == 4) {
                            pb[k] = __builtin_amdgcn_perm(m.lut[k][1], m.lut[k][0], sel) & ~hib;
                        } else {
                            pb[k] = __builtin_amdgcn_perm(m.lut[k][1], m.lut[k][0], sel);
                        }
                    }
                }
#pragma unroll
                for (int k = 0; k < NS; ++k) {
                    Bop[k][q] = (int32_t)pb[k];
                    if (ZS) psum[k] = __builtin_amdgcn_udot4(pb[k] & kmask, 0x01010101u, psum[k], false);
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
                // the tile's output: sum_j P_j of row i0 + r over the four key
                // groups, then the recombined ranges less zp_V sum_j P_j
                const int row = 16 * tile + r;
                if constexpr (WIDE) {
                    uint64_t zterm = 0;
                    if (ZS) {
                        uint64_t p64 = 0;
#pragma unroll
                        for (int k = 0; k < NS; ++k) p64 += (uint64_t)psum[k] << (7 * k);
#pragma unroll
                        for (int x = 16; x <= 32; x *= 2) {
                            const uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)p64, x, 64);
                            const uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(p64 >> 32), x, 64);
                            p64 += ((uint64_t)hi << 32) | lo;
                        }
                        zterm = (uint64_t)(int64_t)a.zp_v * p64;
                    }
                    if (row < a.Lq) {
                        int64_t* orow = reinterpret_cast<int64_t*>(a.out) + (g * a.Lq + row) * (int64_t)d;
#pragma unroll
                        for (int ct = 0; ct < DT; ++ct) {
#pragma unroll
                            for (int t = 0; t < 4; ++t) {
                                uint64_t v = 0;
#pragma unroll
                                for (int k = 0; k < NS; ++k)
                                    v += (uint64_t)(int64_t)acc[ct][k][t] << (7 * k);
                                const int c = 16 * ct + 4 * kq + t;
                                if (c < d) orow[c] = (int64_t)(v - zterm);
                            }
                        }
                    }
                } else {
                    uint32_t zterm = 0;
                    if (ZS) {
                        uint32_t p32 = 0;
#pragma unroll
                        for (int k = 0; k < NS; ++k) p32 += psum[k] << (7 * k);
                        p32 += (uint32_t)__shfl_xor((int)p32, 16, 64);
                        p32 += (uint32_t)__shfl_xor((int)p32, 32, 64);
                        zterm = (uint32_t)a.zp_v * p32;
                    }
                    if (row < a.Lq) {
                        int32_t* orow = reinterpret_cast<int32_t*>(a.out) + (g * a.Lq + row) * (int64_t)d;
#pragma unroll
                        for (int ct = 0; ct < DT; ++ct) {
                            uint32_t res[4];
#pragma unroll
                            for (int t = 0; t < 4; ++t) {
                                uint32_t v = 0;
#pragma unroll
                                for (int k = 0; k < NS; ++k) v += (uint32_t)acc[ct][k][t] << (7 * k);
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
                }
                ks = 0;
                tile += 4;
                rowoff = row_of(tile);
            }
        }
    }

    if constexpr (WIDE) {
        // A code above W somewhere in the unit: every output of the unit again,
        // term by term (V from the staged V^T, codes from memory).
        if (__ballot(floor_seen) != 0 && lane == 0) atomicOr(&s_floor, 1);
        __syncthreads();
        if (s_floor) {
            const uint8_t* cu = a.codes + g * a.Lq * (int64_t)a.ld_codes;
            int64_t* ou = reinterpret_cast<int64_t*>(a.out) + g * a.Lq * (int64_t)d;
            for (int idx = threadIdx.x; idx < a.Lq * d; idx += 256) {
                const int i = idx / d;
                const int c = idx - i * d;
                const uint8_t* crow = cu + (int64_t)i * a.ld_codes;
                uint64_t sum = 0;
                for (int j = 0; j < Lk; ++j) {
                    const int code = BYTES ? crow[j] : (crow[j >> 1] >> (4 * (j & 1))) & 15;
                    const int pos = (j & ~15) + (BYTES ? (j & 15) : av_byte_of_key(j & 15));
                    const int64_t vq = (int64_t)(int8_t)vt[c * m.ldv + pos] - a.zp_v;
                    sum += code <= a.W ? (uint64_t)vq << (a.W - code)
                                       : (uint64_t)(vq >> min(code - a.W, 63));
                }
                ou[(int64_t)i * d + c] = (int64_t)sum;
            }
        }
    }
}

template <int DT, int CB, bool WIDE>
hipError_t launch_cfg(const AvK& a, const AvMfma& m, size_t lds, hipStream_t s) {
    const dim3 grid((unsigned)a.G), block(256);
    if (a.zp_v != 0) launch_kernel(attn_v_mfma_kernel<DT, CB, true, WIDE>, grid, block, lds, s, a, m);
    else launch_kernel(attn_v_mfma_kernel<DT, CB, false, WIDE>, grid, block, lds, s, a, m);
    return hipGetLastError();
}

template <int DT, bool WIDE>
hipError_t launch_cb(int cb, const AvK& a, const AvMfma& m, size_t lds, hipStream_t s) {
    switch (cb) {
        case 1: return launch_cfg<DT, 1, WIDE>(a, m, lds, s);
        case 2: return launch_cfg<DT, 2, WIDE>(a, m, lds, s);
        case 3: return launch_cfg<DT, 3, WIDE>(a, m, lds, s);
        case 4: return launch_cfg<DT, 4, WIDE>(a, m, lds, s);
        case 5: return WIDE ? launch_cfg<DT, 5, true>(a, m, lds, s) : hipErrorNotSupported;
        default: return WIDE ? launch_cfg<DT, 8, true>(a, m, lds, s) : hipErrorNotSupported;
    }
}

// Launch parameters; hipErrorNotSupported for shapes the kernel does not take.
hipError_t launch_any(const AvK& a, int bits, bool wide, hipStream_t stream) {
    AvMfma m;
    m.kp = (a.Lk + 63) / 64 * 64;
    m.nks = m.kp / 64;
    m.ldv = m.kp + 16;
    m.ntiles = (a.Lq + 15) / 16;
    m.vec_out = (a.d % 4 == 0) && ((reinterpret_cast<uintptr_t>(a.out) & 15) == 0);
    m.vec_v = (a.d % 16 == 0) && ((reinterpret_cast<uintptr_t>(a.v) & 15) == 0);
    // the unit's code bytes: rows 0 .. Lq - 1 at stride ld_codes
    const int row_bytes = bits >= 5 ? a.Lk : (a.Lk + 1) / 2;
    const int64_t ub = (int64_t)(a.Lq - 1) * a.ld_codes + row_bytes;
    int dt = 1;
    while (16 * dt < a.d) dt <<= 1;
    const size_t lds = (size_t)16 * dt * m.ldv;
    if (dt > 4 || a.Lk > kAvMfmaMaxLk || ub + 6 > 0x7FFFFFFF || a.G > 0x7FFFFFFF)
        return hipErrorNotSupported;
    m.unit_bytes = (int)ub;
    // nibble codes: P_k byte tables, code c -> 2^(s - 7 k) for 7 k <= s < 7 k + 7,
    // s = W - c
    for (int k = 0; k < 3; ++k) {
        for (int w = 0; w < 4; ++w) m.lut[k][w] = 0;
        for (int c = 0; c < 16 && bits <= 4; ++c) {
            const int s = a.W - c;
            const uint32_t byte = (s >= 7 * k && s < 7 * k + 7) ? (1u << (s - 7 * k)) : 0u;
            m.lut[k][c >> 2] |= byte << (8 * (c & 3));
        }
    }
    const int cb = bits <= 4 ? bits : bits == 5 ? 5 : 8;
    switch (dt) {
        case 1: return wide ? launch_cb<1, true>(cb, a, m, lds, stream)
                            : launch_cb<1, false>(cb, a, m, lds, stream);
        case 2: return wide ? launch_cb<2, true>(cb, a, m, lds, stream)
                            : launch_cb<2, false>(cb, a, m, lds, stream);
        default: return wide ? launch_cb<4, true>(cb, a, m, lds, stream)
                             : launch_cb<4, false>(cb, a, m, lds, stream);
    }
}

}  // namespace
}  // namespace lis

hipError_t launch_attn_v_mfma(const AvArgs& a, hipStream_t stream) {
    const int bits = a.top == 15 ? 4 : a.top == 7 ? 3 : a.top == 3 ? 2 : 1;
    const lis::AvK k{a.codes, a.ld_codes, a.v, a.zp_v, a.G, a.Lq, a.Lk, a.d, a.top, a.out};
    return lis::launch_any(k, bits, false, stream);
}

hipError_t launch_attn_v_wide_mfma(const AvWideArgs& a, hipStream_t stream) {
    const lis::AvK k{a.codes, a.ld_codes, a.v, a.zp_v, a.G, a.Lq, a.Lk, a.d, a.W, a.out};
    return lis::launch_any(k, a.bits, true, stream);
}

}  // namespace fqvit
