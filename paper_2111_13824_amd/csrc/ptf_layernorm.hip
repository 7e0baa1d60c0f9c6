// Integer-only PTF LayerNorm for gfx950 (Sec. 3.2 phase-1 shift; Supplement
// A.1 statistics, A/B factors, dyadic N2/2^N1 form and output Y_Q).
//
// Per token row: X^ = (X_Q - zp) << alpha, M1 = sum X^, M2 = sum X^^2,
// V = C M2 - M1^2 (exact integers); in IEEE double D = sqrt(V), r = C/D,
// m = M1/D; per element A = gs r, B = bs - gs m with gs = gamma/s_out,
// bs = beta/s_out; N1 = clamp(b - 1 - floor(log2|A|), 0, 30),
// N2 = min(floor(|A| 2^N1), 2^31 - 1); Y = clip(floor((sign(A) N2 X^ +
// rint(B 2^N1) + 2^(N1-1)) / 2^N1) + zp_out).
//
// The last step is evaluated as floor(At * X^ + (Bg + 1/2)) in double with
// At = sign(A) N2 2^-N1 and Bg = rint(B 2^N1) 2^-N1.  Every term is an exact
// dyadic rational: At X^ has at most 31 + 15 significant bits, Bg + 1/2 and the
// sum are multiples of 2^-N1 below 2^53 2^-N1 whenever |rint(B 2^N1)| < 2^52,
// so the fused multiply-add rounds nothing.  Larger B saturate the output
// whatever the rounding.  The whole file is compiled with -ffp-contract=off so
// that A and B are each rounded exactly as written.
//
// Kernels: ln_rows_kernel (256 <= C <= 1024: a wavefront per row, batches of
// rows), ln_seg_kernel (C < 256: L lanes per row, the factors of several rows
// computed together), ln_fast_kernel (other aligned shapes: L lanes per row,
// per-channel gs, bs and shifts held in registers) and ln_generic_kernel (any
// C and alignment).  In each, a lane owns whole 4-channel dwords of a row, so
// that loads and stores are coalesced dwords and the row statistics are
// shuffle reductions.
#include <climits>

#include "fqvit_launch.h"

namespace fqvit {
namespace {

constexpr int kBlock = 256;

// Output of one element on the int8 container grid.
__device__ __forceinline__ int ln_requant(double A, double B, int xh, int bits, int zp_out,
                                          int qlo, int qhi) {
    const int e = __builtin_amdgcn_frexp_exp(A);          // |A| = f 2^e, f in [0.5, 1)
    int N1 = min(max(bits - e, 0), 30);                   // b - 1 - floor(log2 |A|)
    N1 = (A == 0.0) ? 0 : N1;
    const double N2 = fmin(floor(ldexp(fabs(A), N1)), 2147483647.0);
    const double At = ldexp(copysign(N2, A), -N1);
    const double Bg = ldexp(rint(ldexp(B, N1)), -N1);
    const double val = fma(At, (double)xh, Bg + 0.5);
    const double w = fmin(fmax(floor(val), -1024.0), 1024.0);
    return min(max((int)w + zp_out, qlo), qhi);
}

template <typename T>
__device__ __forceinline__ T seg_sum(T v, int L) {
    for (int off = 1; off < L; off <<= 1) v += __shfl_xor(v, off, 64);
    return v;
}

// Sum over aligned segments of L lanes (L a power of two <= 64), result in
// every lane of the segment.  Within a row of 16 lanes: DPP quad permutes
// (xor 1, xor 2), then half-row and row mirrors, each of which pairs lanes
// whose partial sums are already equal across the group they stand for.
// Across rows: readlane of the row totals.
__device__ __forceinline__ int dpp_seg_sum(int v, int L) {
    if (L >= 2) v += __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false);   // quad_perm 1,0,3,2
    if (L >= 4) v += __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false);   // quad_perm 2,3,0,1
    if (L >= 8) v += __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false);  // row_half_mirror
    if (L >= 16) v += __builtin_amdgcn_update_dpp(0, v, 0x140, 0xF, 0xF, false); // row_mirror
    if (L >= 32) {
        const int r0 = __builtin_amdgcn_readlane(v, 0), r1 = __builtin_amdgcn_readlane(v, 16);
        const int r2 = __builtin_amdgcn_readlane(v, 32), r3 = __builtin_amdgcn_readlane(v, 48);
        if (L == 64) {
            v = r0 + r1 + r2 + r3;
        } else {
            v = ((threadIdx.x & 63) < 32) ? r0 + r1 : r2 + r3;
        }
    }
    return v;
}

// Per-row factors: r = C / sqrt(V), m = M1 / sqrt(V); both 0 for V = 0.
__device__ __forceinline__ void row_factors(int64_t m1, int64_t m2, int C, double& r,
                                            double& m) {
    const int64_t V = (int64_t)C * m2 - m1 * m1;
    r = 0.0;
    m = 0.0;
    if (V > 0) {
        const double D = sqrt((double)V);
        r = (double)C / D;
        m = (double)m1 / D;
    }
}

typedef short short2_t __attribute__((ext_vector_type(2)));

// Output of one element when A = gs r is known to lie in [2^(b-31), 2^b): then
// N1 = b - 1 - floor(log2 |A|) needs no clamp and sign(A) N2 / 2^N1 is A with
// its significand cut to b bits, a mask on the high word (b <= 8 keeps the
// low word zero).  rint(B 2^N1) 2^-N1 is B rounded to the grid of that last
// bit, 2^(E - b + 1) with E the exponent of A, ties to even: adding and
// subtracting M = 1.5 2^(E - b + 53) does exactly that while |B| < 2^(E - b + 52);
// larger B (and the oracle's clamp of B 2^N1 at 2^62) saturate the output
// either way, since |A X^| < 2^(E + 12).  Same result as ln_requant.
// m_add = (53 - b) << 20 | 0x80000 builds M's high word from A's exponent
// field.  With c = zp_out + 1/2 + 512, v = At X^ + (Bg + c) is exact and
// floor(v) = Y + 512 when unclamped; v_cvt_i32_f64 truncates (floor for
// v >= 0) and saturates, and the clamp to [lo, hi] = [qlo + 512, qhi + 512]
// (both positive, so a negative v lands on the lower bound either way)
// returns Y + 512, whose low byte is Y's.
__device__ __forceinline__ int ln_requant_rows(double A, double B, int xh, uint32_t hi_mask,
                                               uint32_t m_add, double c, int lo, int hi) {
    const uint32_t hiA = (uint32_t)((uint64_t)__double_as_longlong(A) >> 32);
    const double At = __longlong_as_double((int64_t)((uint64_t)(hiA & hi_mask) << 32));
    const double M = __longlong_as_double((int64_t)((uint64_t)((hiA & 0x7FF00000u) + m_add) << 32));
    const double Bc = ((B + M) - M) + c;
    const double v = fma(At, (double)xh, Bc);
    int q;
    asm("v_cvt_i32_f64 %0, %1" : "=v"(q) : "v"(v));
    asm("v_med3_i32 %0, %1, %2, %3" : "=v"(q) : "v"(q), "s"(lo), "v"(hi));
    return q;
}

// Fast path: C % 4 == 0, dword-aligned rows, W dwords per lane (W <= 8).
// WIDE selects 64-bit per-lane sums of squares (K >= 6).
template <int W, bool WIDE>
__global__ __launch_bounds__(kBlock) void ln_fast_kernel(LnArgs a, int lshift) {
    extern __shared__ double smem[];
    const int nd = a.C >> 2;
    // LDS layout [b][dword]: lane li reads entry (b, li + L w), so the lanes of
    // a wavefront read consecutive entries.
    double* s_gs = smem;
    double* s_bs = smem + a.C;
    int* s_sh = reinterpret_cast<int*>(smem + 2 * a.C);
    __shared__ double s_ext[2][kBlock / 64];
    __shared__ int s_zero[kBlock / 64];
    double gmax = 0.0, gmin = INFINITY;
    int anyzero = 0;
    for (int c = threadIdx.x; c < a.C; c += blockDim.x) {
        const int e = (c & 3) * nd + (c >> 2);
        const double gs = (double)a.gamma[c] / (double)a.s_out;
        s_gs[e] = gs;
        s_bs[e] = (double)a.beta[c] / (double)a.s_out;
        s_sh[e] = min((int)a.alpha[c], a.K);
        const double ag = fabs(gs);
        gmax = fmax(gmax, ag);
        if (ag == 0.0) anyzero = 1; else gmin = fmin(gmin, ag);
    }
    for (int off = 1; off < 64; off <<= 1) {
        gmax = fmax(gmax, __shfl_xor(gmax, off, 64));
        gmin = fmin(gmin, __shfl_xor(gmin, off, 64));
        anyzero |= __shfl_xor(anyzero, off, 64);
    }
    if ((threadIdx.x & 63) == 0) {
        s_ext[0][threadIdx.x >> 6] = gmax;
        s_ext[1][threadIdx.x >> 6] = gmin;
        s_zero[threadIdx.x >> 6] = anyzero;
    }
    __syncthreads();
    for (int w = 0; w < (int)(blockDim.x >> 6); ++w) {
        gmax = fmax(gmax, s_ext[0][w]);
        gmin = fmin(gmin, s_ext[1][w]);
        anyzero |= s_zero[w];
    }

    const int lane = threadIdx.x & 63;
    const int L = 1 << lshift;
    const int seg = lane >> lshift;
    const int li = lane & (L - 1);
    const int R = 64 >> lshift;

    double gs[4 * W], bs[4 * W];
    int mul[4 * W];
    bool ok[W];
#pragma unroll
    for (int w = 0; w < W; ++w) {
        const int dw = li + (w << lshift);
        ok[w] = dw < nd;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            const int e = ok[w] ? b * nd + dw : 0;
            gs[4 * w + b] = s_gs[e];
            bs[4 * w + b] = s_bs[e];
            mul[4 * w + b] = ok[w] ? 1 << s_sh[e] : 0;
        }
    }

    // packed-statistics constants per dword (u = zp_in + 128): i16 pairs of
    // 2^alpha and of -u 2^alpha, bytes of 2^alpha, and sum -u 2^alpha
    uint32_t mulp[2 * W], zmp[2 * W], mulb[W];
    uint32_t m1init = 0;
    const int u_in = a.zp_in + 128;
#pragma unroll
    for (int w = 0; w < W; ++w) {
        mulb[w] = 0;
        mulp[2 * w] = mulp[2 * w + 1] = 0;
        zmp[2 * w] = zmp[2 * w + 1] = 0;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            const uint32_t mb = (uint32_t)mul[4 * w + b];              // 0 past C
            const uint32_t zm = (uint32_t)(-u_in) * mb;
            mulb[w] |= mb << (8 * b);
            mulp[2 * w + (b >> 1)] |= mb << (16 * (b & 1));
            zmp[2 * w + (b >> 1)] |= (zm & 0xFFFFu) << (16 * (b & 1));
            m1init += zm;
        }
    }

    const int qlo = -(1 << (a.bits - 1));
    const int qhi = (1 << (a.bits - 1)) - 1;
    const uint32_t hi_mask = ~((1u << (21 - a.bits)) - 1u);   // keep sign, exponent, b-1 bits
    // one opaque scalar, so that the exponent add stays one instruction
    uint32_t m_add = ((uint32_t)(53 - a.bits) << 20) | 0x80000u;
    asm volatile("" : "+s"(m_add));
    const double amax = ldexp(1.0, a.bits), amin = ldexp(1.0, a.bits - 31);
    const double cadd = (double)a.zp_out + 512.5;
    const int lo512 = qlo + 512, hi512 = qhi + 512;
    const int64_t gw = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    const int64_t nw = ((int64_t)gridDim.x * blockDim.x) >> 6;

    int64_t r0 = gw * R;
    uint32_t xn[W];
    {
        const int64_t row = r0 + seg;
        const uint32_t* xr = reinterpret_cast<const uint32_t*>(a.x + (row < a.T ? row : 0) * a.C);
#pragma unroll
        for (int w = 0; w < W; ++w) xn[w] = ok[w] ? __builtin_nontemporal_load(xr + li + (w << lshift)) : 0u;
    }
    for (; r0 < a.T; r0 += nw * R) {
        const int64_t row = r0 + seg;
        const bool rok = row < a.T;
        const int64_t rr = rok ? row : 0;
        uint32_t xv[W];
#pragma unroll
        for (int w = 0; w < W; ++w) xv[w] = xn[w];
        {   // prefetch the next row of this lane
            const int64_t nrow = r0 + nw * R + seg;
            const uint32_t* xr = reinterpret_cast<const uint32_t*>(a.x + (nrow < a.T ? nrow : 0) * a.C);
#pragma unroll
            for (int w = 0; w < W; ++w)
                xn[w] = (ok[w] && r0 + nw * R < a.T) ? __builtin_nontemporal_load(xr + li + (w << lshift)) : 0u;
        }

        int xh[4 * W];
        int64_t M1, M2;
        if (WIDE) {
            int m1 = 0;
            int64_t m2w = 0;
#pragma unroll
            for (int w = 0; w < W; ++w) {
#pragma unroll
                for (int b = 0; b < 4; ++b) {
                    const int x = (int)(int8_t)(xv[w] >> (8 * b));
                    const int h = __mul24(x - a.zp_in, mul[4 * w + b]);   // 0 past C
                    xh[4 * w + b] = h;
                    m1 += h;
                    m2w += (int64_t)h * h;
                }
            }
            M1 = seg_sum<int>(m1, L);
            M2 = seg_sum<int64_t>(m2w, L);
        } else {
            // packed i16 X^ pairs, M1 by byte dot products, M2 by i16 pair dot
            // products (as in the row-batch kernel; exact, |X^| < 2^15)
            uint32_t m1 = m1init, m2 = 0;
#pragma unroll
            for (int w = 0; w < W; ++w) {
                const uint32_t xu = xv[w] ^ 0x80808080u;
                const uint32_t p0 = __builtin_amdgcn_perm(xu, xu, 0x0C010C00u);
                const uint32_t p1 = __builtin_amdgcn_perm(xu, xu, 0x0C030C02u);
                const short2_t h0 = __builtin_bit_cast(short2_t, p0) * __builtin_bit_cast(short2_t, mulp[2 * w]) +
                                    __builtin_bit_cast(short2_t, zmp[2 * w]);
                const short2_t h1 = __builtin_bit_cast(short2_t, p1) * __builtin_bit_cast(short2_t, mulp[2 * w + 1]) +
                                    __builtin_bit_cast(short2_t, zmp[2 * w + 1]);
                m1 = __builtin_amdgcn_udot4(xu, mulb[w], m1, false);
                m2 = (uint32_t)__builtin_amdgcn_sdot2(h0, h0, (int)m2, false);
                m2 = (uint32_t)__builtin_amdgcn_sdot2(h1, h1, (int)m2, false);
                xh[4 * w + 0] = h0.x;
                xh[4 * w + 1] = h0.y;
                xh[4 * w + 2] = h1.x;
                xh[4 * w + 3] = h1.y;
            }
            // per-lane m2 < 2^31: sum its 16-bit halves separately in 32 bits
            M1 = dpp_seg_sum((int)m1, L);
            const int lo = dpp_seg_sum((int)(m2 & 0xFFFFu), L);
            const int hi = dpp_seg_sum((int)(m2 >> 16), L);
            M2 = ((int64_t)hi << 16) + lo;
        }
        double r, m;
        row_factors(M1, M2, a.C, r, m);
        const bool fast = r > 0.0 && !anyzero && gmax * r < amax && gmin * r >= amin;

        uint32_t* yr = reinterpret_cast<uint32_t*>(a.y + rr * a.C);
        if (fast) {
#pragma unroll
            for (int w = 0; w < W; ++w) {
                int q[4];
#pragma unroll
                for (int b = 0; b < 4; ++b) {
                    const int k = 4 * w + b;
                    const double A = gs[k] * r;
                    const double B = bs[k] - gs[k] * m;
                    q[b] = ln_requant_rows(A, B, xh[k], hi_mask, m_add, cadd, lo512, hi512);
                }
                // the low bytes of Y + 512 are Y's
                const uint32_t lo = __builtin_amdgcn_perm((uint32_t)q[1], (uint32_t)q[0], 0x0C0C0400u);
                const uint32_t hi = __builtin_amdgcn_perm((uint32_t)q[3], (uint32_t)q[2], 0x0C0C0400u);
                const uint32_t pack = __builtin_amdgcn_perm(hi, lo, 0x05040100u);
                if (rok && ok[w]) __builtin_nontemporal_store(pack, yr + li + (w << lshift));
            }
        } else {
#pragma unroll
            for (int w = 0; w < W; ++w) {
                uint32_t pack = 0;
#pragma unroll
                for (int b = 0; b < 4; ++b) {
                    const int k = 4 * w + b;
                    const double A = gs[k] * r;
                    const double B = bs[k] - gs[k] * m;
                    const int q = ln_requant(A, B, xh[k], a.bits, a.zp_out, qlo, qhi);
                    pack |= ((uint32_t)q & 0xFFu) << (8 * b);
                }
                if (rok && ok[w]) __builtin_nontemporal_store(pack, yr + li + (w << lshift));
            }
        }
    }
}

// General path: any C in [1, 8192], any alignment.  One wavefront per row,
// two passes over the row (the second from cache), per-channel factors
// computed in place.
__global__ __launch_bounds__(kBlock) void ln_generic_kernel(LnArgs a) {
    const int lane = threadIdx.x & 63;
    const int64_t gw = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    const int64_t nw = ((int64_t)gridDim.x * blockDim.x) >> 6;
    const int qlo = -(1 << (a.bits - 1));
    const int qhi = (1 << (a.bits - 1)) - 1;
    for (int64_t row = gw; row < a.T; row += nw) {
        const int8_t* xr = a.x + row * a.C;
        int64_t m1 = 0, m2 = 0;
        for (int c = lane; c < a.C; c += 64) {
            const int64_t h = (int64_t)((int)xr[c] - a.zp_in) * ((int64_t)1 << min((int)a.alpha[c], a.K));
            m1 += h;
            m2 += h * h;
        }
        for (int off = 1; off < 64; off <<= 1) {
            m1 += __shfl_xor(m1, off, 64);
            m2 += __shfl_xor(m2, off, 64);
        }
        double r, m;
        row_factors(m1, m2, a.C, r, m);
        int8_t* yr = a.y + row * a.C;
        for (int c = lane; c < a.C; c += 64) {
            const int h = ((int)xr[c] - a.zp_in) * (1 << min((int)a.alpha[c], a.K));
            const double gs = (double)a.gamma[c] / (double)a.s_out;
            const double bs = (double)a.beta[c] / (double)a.s_out;
            const double A = gs * r;
            const double B = bs - gs * m;
            yr[c] = (int8_t)ln_requant(A, B, h, a.bits, a.zp_out, qlo, qhi);
        }
    }
}

// ---------------------------------------------------------------------------
// Row-batch kernel for rows of 256..1024 channels (C % 4 == 0, dword-aligned)
// whose sums of squares fit 32 bits (C (255 2^K)^2 < 2^32).
//
// A wavefront owns a contiguous run of rows, taken R = 1, 2 or 4 at a time (a
// batch); lane l owns dwords l, l + 64, ... of each row (coalesced dword loads
// and stores).  The
// per-channel (gs, bs) pairs stay in LDS in [byte][dword] order, so that the
// 16-byte reads of a wavefront are consecutive.  Per dword, with xu = x + 128 (the byte with
// its sign bit flipped, 0..255) and u = zp_in + 128:
//   X^ pairs  = (xu pairs) * (2^alpha pairs) + (-u 2^alpha pairs)   packed i16,
//               exact: |X^| <= 255 2^7 < 2^15
//   M1 lane  += dot4(xu bytes, 2^alpha bytes), the -u sum_c 2^alpha part of
//               every row being a per-lane constant
//   M2 lane  += dot2(X^ pair, X^ pair), twice
// The R x 2 per-row totals are reduced together: a 32-lane swap-add and a
// 16-lane swap-add leave row j's partial sums in lane group j (64 / R lanes
// from lane 64 j / R), four row rotations finish them, and one evaluation of
// the square root and the two divisions serves the R rows.  The per-row
// factors reach every lane as scalars.
//
// Output, when the row's factors fit (see ln_requant_rows): with
// c = zp_out + 1/2 + 512, v = At X^ + (Bg + c) is exact (multiples of 2^-N1
// below 2^53 2^-N1) and floor(v) = w + zp_out + 512; v_cvt_i32_f64 truncates
// (floor for v >= 0) and saturates, and a clamp to [qlo + 512, qhi + 512]
// (both positive, so a negative v lands on the lower bound either way) gives
// Y + 512, whose low byte is Y's.

__device__ __forceinline__ uint32_t swap_add32(uint32_t a, uint32_t b) {
    // lanes 0-31: a summed over lanes l and l + 32; lanes 32-63: the same for b
    const auto s = __builtin_amdgcn_permlane32_swap(a, b, false, false);
    return s[0] + s[1];
}

__device__ __forceinline__ uint32_t swap_add16(uint32_t a, uint32_t b) {
    // within each 32-lane half: lanes 0-15 a, lanes 16-31 b, summed over
    // lanes l and l + 16
    const auto s = __builtin_amdgcn_permlane16_swap(a, b, false, false);
    return s[0] + s[1];
}

__device__ __forceinline__ uint32_t row16_sum(uint32_t v) {
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x128, 0xF, 0xF, false);  // row_ror:8
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x124, 0xF, 0xF, false);  // row_ror:4
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x122, 0xF, 0xF, false);  // row_ror:2
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x121, 0xF, 0xF, false);  // row_ror:1
    return v;
}

typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x3_t __attribute__((ext_vector_type(3)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ double readlane_f64(double v, int lane) {
    const uint64_t b = (uint64_t)__double_as_longlong(v);
    const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)b, lane);
    const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(b >> 32), lane);
    return __longlong_as_double((int64_t)(((uint64_t)hi << 32) | lo));
}

// Rows r0 .. r0 + nr - 1 of the lane's dwords (zeros elsewhere; nr may be 0),
// as buffer loads through the descriptor of the whole input: the loads that
// are not needed address past its end and return 0 without a memory access,
// so every load is issued unconditionally and the compiler can count the
// loads in flight across the batches.
// CT: lane l holds dwords W l .. W l + W - 1 of a row (nd = 64 W): one load
// of 4 W bytes per lane and row.
template <int W, int R, bool CT>
__device__ __forceinline__ void load_rows(uint32_t (&xv)[R][W],
                                          __amdgpu_buffer_rsrc_t xr, int64_t r0, int nr, int nd,
                                          int lane, const bool (&ok)[W]) {
    if constexpr (CT) {
#pragma unroll
        for (int j = 0; j < R; ++j) {
            const int off = j < nr ? (int)(((r0 + j) * nd + W * lane) * 4) : INT_MIN;
            if constexpr (W == 1) {
                xv[j][0] = __builtin_amdgcn_raw_buffer_load_b32(xr, off, 0, 0);
            } else if constexpr (W == 2) {
                const u32x2_t v = __builtin_amdgcn_raw_buffer_load_b64(xr, off, 0, 0);
                xv[j][0] = v[0]; xv[j][1] = v[1];
            } else if constexpr (W == 3) {
                const u32x3_t v = __builtin_amdgcn_raw_buffer_load_b96(xr, off, 0, 0);
                xv[j][0] = v[0]; xv[j][1] = v[1]; xv[j][2] = v[2];
            } else {
                const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(xr, off, 0, 0);
                xv[j][0] = v[0]; xv[j][1] = v[1]; xv[j][2] = v[2]; xv[j][3] = v[3];
            }
        }
        return;
    }
#pragma unroll
    for (int j = 0; j < R; ++j) {
#pragma unroll
        for (int w = 0; w < W; ++w) {
            const int off = (j < nr && ok[w]) ? (int)(((r0 + j) * nd + lane + 64 * w) * 4) : INT_MIN;
            // default cache policy: streaming (non-temporal) loads measured
            // 0.1-0.5 us slower on the ViT-B, ViT-L and Swin-S rows
            xv[j][w] = __builtin_amdgcn_raw_buffer_load_b32(xr, off, 0, 0);
        }
    }
}

// Per-lane constants of the row-batch kernel (see ln_rows_kernel).
template <int W>
struct RowsCtx {
    uint32_t mulp[2 * W], zmp[2 * W], mulb[W];
    uint32_t m1init;
    double gmaxl, gminl;
    bool zerol;
    bool ok[W];
    uint32_t hi_mask, m_add;
    double amax, amin, cadd;
    int lo512, hi512, qlo, qhi;
};

// Statistics of rows r0 .. r0 + nr - 1 (nr in 1..R) from their dwords xv: the
// packed X^ of each row, and the factors r, m of row j in lane group j.
template <int W, int R>
struct RowsStats {
    uint32_t hp[R][2 * W];
    double r, m;
};

// Lane group j's totals of row j: v[j] summed over the wavefront, for R rows.
template <int R>
__device__ __forceinline__ uint32_t rows_total(const uint32_t (&v)[R]) {
    if constexpr (R == 4) return row16_sum(swap_add16(swap_add32(v[0], v[2]), swap_add32(v[1], v[3])));
    else if constexpr (R == 2) {
        const uint32_t h = swap_add32(v[0], v[1]);   // row j in lanes 32 j .. 32 j + 31
        return row16_sum(swap_add16(h, h));
    } else {
        const uint32_t h = swap_add32(v[0], v[0]);
        return row16_sum(swap_add16(h, h));
    }
}

template <int W, int R>
__device__ __forceinline__ void rows_stats(const LnArgs& a, const RowsCtx<W>& k,
                                           const uint32_t (&xv)[R][W], RowsStats<W, R>& st) {
    uint32_t m1[R], m2[R];
#pragma unroll
    for (int j = 0; j < R; ++j) {
        m1[j] = k.m1init;
        m2[j] = 0;
#pragma unroll
        for (int w = 0; w < W; ++w) {
            const uint32_t xu = xv[j][w] ^ 0x80808080u;
            const uint32_t p0 = __builtin_amdgcn_perm(xu, xu, 0x0C010C00u);
            const uint32_t p1 = __builtin_amdgcn_perm(xu, xu, 0x0C030C02u);
            const short2_t h0 = __builtin_bit_cast(short2_t, p0) * __builtin_bit_cast(short2_t, k.mulp[2 * w]) +
                                __builtin_bit_cast(short2_t, k.zmp[2 * w]);
            const short2_t h1 = __builtin_bit_cast(short2_t, p1) * __builtin_bit_cast(short2_t, k.mulp[2 * w + 1]) +
                                __builtin_bit_cast(short2_t, k.zmp[2 * w + 1]);
            m1[j] = __builtin_amdgcn_udot4(xu, k.mulb[w], m1[j], false);
            m2[j] = (uint32_t)__builtin_amdgcn_sdot2(h0, h0, (int)m2[j], false);
            m2[j] = (uint32_t)__builtin_amdgcn_sdot2(h1, h1, (int)m2[j], false);
            st.hp[j][2 * w] = __builtin_bit_cast(uint32_t, h0);
            st.hp[j][2 * w + 1] = __builtin_bit_cast(uint32_t, h1);
        }
    }
    const uint32_t t1 = rows_total<R>(m1);
    const uint32_t t2 = rows_total<R>(m2);
    row_factors((int64_t)(int32_t)t1, (int64_t)t2, a.C, st.r, st.m);
}

// Output of the batch.  A row whose factors are in the fast range is packed
// into bytes and stored as soon as it is computed, so that the stores of a
// wavefront spread over its arithmetic instead of leaving together at its end;
// the other rows are written element by element (their bytes read again).
template <int W, int R, bool CT>
__device__ __forceinline__ void rows_output(const LnArgs& a, const RowsCtx<W>& k,
                                            const double2* s_gb, const RowsStats<W, R>& st,
                                            int64_t r0, int nr, int nd, int lane,
                                            uint32_t* y32, __amdgpu_buffer_rsrc_t yr_rsrc) {
#pragma unroll
    for (int j = 0; j < R; ++j) {
        if (j >= nr) break;
        const double rj = readlane_f64(st.r, (64 / R) * j);
        const double mj = readlane_f64(st.m, (64 / R) * j);
        const bool lane_fits = !k.zerol && k.gmaxl * rj < k.amax && k.gminl * rj >= k.amin;
        if (rj > 0.0 && __ballot(!lane_fits) == 0) {
            uint32_t yo[W];
#pragma unroll
            for (int w = 0; w < W; ++w) {
                int q[4];
#pragma unroll
                for (int b = 0; b < 4; ++b) {
                    const uint32_t hw = st.hp[j][2 * w + (b >> 1)];
                    const int xh = (b & 1) ? (int)hw >> 16 : (int)(int16_t)(hw & 0xFFFFu);
                    const double2 gb = s_gb[b * nd + (k.ok[w] ? lane + 64 * w : 0)];
                    const double A = gb.x * rj;
                    const double B = gb.y - gb.x * mj;
                    q[b] = ln_requant_rows(A, B, xh, k.hi_mask, k.m_add, k.cadd, k.lo512, k.hi512);
                }
                const uint32_t lo = __builtin_amdgcn_perm((uint32_t)q[1], (uint32_t)q[0], 0x0C0C0400u);
                const uint32_t hi = __builtin_amdgcn_perm((uint32_t)q[3], (uint32_t)q[2], 0x0C0C0400u);
                yo[w] = __builtin_amdgcn_perm(hi, lo, 0x05040100u);
                // one dword at a time: the f64 temporaries of all 4 W
                // elements would not fit the register budget
                __builtin_amdgcn_sched_barrier(0);
            }
            if constexpr (CT) {
                const int off = (int)(((r0 + j) * nd + W * lane) * 4);
                if constexpr (W == 1) {
                    __builtin_amdgcn_raw_buffer_store_b32(yo[0], yr_rsrc, off, 0, 2);
                } else if constexpr (W == 2) {
                    __builtin_amdgcn_raw_buffer_store_b64(u32x2_t{yo[0], yo[1]}, yr_rsrc, off, 0, 2);
                } else if constexpr (W == 3) {
                    __builtin_amdgcn_raw_buffer_store_b96(u32x3_t{yo[0], yo[1], yo[2]}, yr_rsrc, off, 0, 2);
                } else {
                    __builtin_amdgcn_raw_buffer_store_b128(u32x4_t{yo[0], yo[1], yo[2], yo[3]}, yr_rsrc, off, 0, 2);
                }
            } else {
                uint32_t* yr = y32 + (r0 + j) * nd + lane;
#pragma unroll
                for (int w = 0; w < W; ++w)
                    if (k.ok[w]) __builtin_nontemporal_store(yo[w], yr + 64 * w);
            }
        } else {
            const int8_t* xrow = a.x + (r0 + j) * a.C;
            int8_t* yrow = a.y + (r0 + j) * a.C;
#pragma unroll 1
            for (int c = lane; c < a.C; c += 64) {
                const int xh = ((int)xrow[c] - a.zp_in) * (1 << min((int)a.alpha[c], a.K));
                const int dq = c >> 2;
                const double2 gb = s_gb[(c & 3) * nd + (CT ? (dq % W) * 64 + dq / W : dq)];
                const double A = gb.x * rj;
                const double B = gb.y - gb.x * mj;
                yrow[c] = (int8_t)ln_requant(A, B, xh, a.bits, a.zp_out, k.qlo, k.qhi);
            }
        }
    }
}

// A wavefront owns a contiguous run of rows and takes them NB batches of R rows
// at a time: the loads of all NB batches are issued first, then the batches
// are computed in order, so the loads of the later ones stream in under the
// arithmetic of the earlier ones.  No load is in flight across the loop's
// back edge (a wait there would cover every outstanding load).  BLOCK threads
// per workgroup; the grid sets the number of wavefronts per CU.
template <int W, int R, int BLOCK, int NB, bool CT>
__global__ __launch_bounds__(BLOCK) void ln_rows_kernel(LnArgs a) {
    extern __shared__ double smem[];
    double2* s_gb = reinterpret_cast<double2*>(smem);        // (gs, bs) at [b][dword]
    uint4* s_pk = reinterpret_cast<uint4*>(s_gb + a.C);      // per dword, see below
    const int nd = a.C >> 2;
    const int lane = threadIdx.x & 63;
    uint32_t* y32 = reinterpret_cast<uint32_t*>(a.y);

    // Contiguous run of rows of this wavefront.  Wavefronts are numbered
    // across workgroups first, so that the ones with an extra row (the
    // remainder of T / nw) spread over all CUs.
    constexpr int kWaves = BLOCK / 64;
    const int64_t nw = (int64_t)gridDim.x * kWaves;
    const int64_t gw = (int64_t)__builtin_amdgcn_readfirstlane(threadIdx.x >> 6) * gridDim.x +
                       blockIdx.x;
    // the whole input, a.T * a.C < 2^31 bytes (checked by the launcher)
    const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
        (void*)a.x, (short)0, (int)(a.T * a.C), 0x00020000);
    const __amdgpu_buffer_rsrc_t yrs = __builtin_amdgcn_make_buffer_rsrc(
        (void*)a.y, (short)0, (int)(a.T * a.C), 0x00020000);
    const int64_t base = a.T / nw, rem = a.T % nw;
    int64_t ra = gw * base + min(gw, rem);
    const int64_t r1 = ra + base + (gw < rem ? 1 : 0);
    RowsCtx<W> k;
#pragma unroll
    for (int w = 0; w < W; ++w) k.ok[w] = CT || lane + 64 * w < nd;

    // Set-up, one thread per dword (4 channels; nd <= 256 <= blockDim): its
    // loads go first, then the first two batches of rows, so that the
    // per-channel factors are computed while the rows stream in.
    //   gs = gamma / s_out, bs = beta / s_out (binary64), and per-dword
    //   constants with u = zp_in + 128:
    //   s_pk[2 dw]     = i16 pairs of 2^alpha (channels 0,1 and 2,3),
    //                    i16 pairs of -u 2^alpha (same order)
    //   s_pk[2 dw + 1] = bytes of 2^alpha, sum of -u 2^alpha, and the largest
    //                    and smallest high word of |gs| over the 4 channels
    const int sdw = threadIdx.x;
    // LDS position of dword sdw: CT keeps the constants of the dwords a lane
    // holds (W l + w) at w 64 + l, so the reads stay lane-consecutive
    const int spos = CT ? (sdw % W) * 64 + sdw / W : sdw;
    float sg[4], sb[4];
    int sa[4];
    if (sdw < nd) {
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            sg[b] = a.gamma[4 * sdw + b];
            sb[b] = a.beta[4 * sdw + b];
            sa[b] = a.alpha[4 * sdw + b];
        }
    }
    uint32_t xv[NB][R][W];
    int nr[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) {
        nr[i] = (int)max<int64_t>(0, min<int64_t>(R, r1 - ra - R * i));
        load_rows<W, R, CT>(xv[i], xr, ra + R * i, nr[i], nd, lane, k.ok);
    }

    const int u = a.zp_in + 128;
    if (sdw < nd) {
        uint32_t mulp[2] = {0, 0}, zmp[2] = {0, 0}, mulb = 0, m1p = 0, ghi = 0, glo = 0x7FF00000u;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            const double gs = (double)sg[b] / (double)a.s_out;
            s_gb[b * nd + spos] = double2{gs, (double)sb[b] / (double)a.s_out};
            const int sh = min(sa[b], a.K);
            const uint32_t zm = (uint32_t)(-u) << sh;
            mulb |= (1u << sh) << (8 * b);
            mulp[b >> 1] |= (1u << sh) << (16 * (b & 1));
            zmp[b >> 1] |= (zm & 0xFFFFu) << (16 * (b & 1));
            m1p += zm;
            const uint32_t h = (uint32_t)((uint64_t)__double_as_longlong(gs) >> 32) & 0x7FFFFFFFu;
            ghi = max(ghi, h);
            glo = min(glo, h);
        }
        s_pk[2 * spos] = uint4{mulp[0], mulp[1], zmp[0], zmp[1]};
        s_pk[2 * spos + 1] = uint4{mulb, m1p, ghi, glo};
    }
    __syncthreads();
    if (nr[0] <= 0) return;

    uint32_t ghi = 0, glo = 0x7FF00000u;
    k.m1init = 0;
#pragma unroll
    for (int w = 0; w < W; ++w) {
        const int dw = k.ok[w] ? lane + 64 * w : 0;
        const uint4 p = s_pk[2 * dw];
        const uint4 q = s_pk[2 * dw + 1];
        k.mulp[2 * w] = k.ok[w] ? p.x : 0u;
        k.mulp[2 * w + 1] = k.ok[w] ? p.y : 0u;
        k.zmp[2 * w] = k.ok[w] ? p.z : 0u;
        k.zmp[2 * w + 1] = k.ok[w] ? p.w : 0u;
        k.mulb[w] = k.ok[w] ? q.x : 0u;
        k.m1init += k.ok[w] ? q.y : 0u;
        ghi = k.ok[w] ? max(ghi, q.z) : ghi;
        glo = k.ok[w] ? min(glo, q.w) : glo;
    }
    // Bounds on |gs| over the lane's channels from the high words alone
    // (|gs| <= gmaxl, |gs| >= gminl; a row whose factors come that close to a
    // bound of the fast range takes the general path).  Zero or subnormal
    // gs (high word 0) always takes the general path.
    k.gmaxl = __longlong_as_double((int64_t)(((uint64_t)ghi << 32) | 0xFFFFFFFFu));
    k.gminl = __longlong_as_double((int64_t)((uint64_t)glo << 32));
    k.zerol = glo == 0;

    k.qlo = -(1 << (a.bits - 1));
    k.qhi = (1 << (a.bits - 1)) - 1;
    k.hi_mask = ~((1u << (21 - a.bits)) - 1u);
    // one opaque scalar, so that the exponent add stays one instruction (the
    // compiler would otherwise split the constant into a subtract and an add)
    uint32_t m_add = ((uint32_t)(53 - a.bits) << 20) | 0x80000u;
    asm volatile("" : "+s"(m_add));
    k.m_add = m_add;
    k.amax = ldexp(1.0, a.bits);
    k.amin = ldexp(1.0, a.bits - 31);
    k.cadd = (double)a.zp_out + 512.5;
    k.lo512 = k.qlo + 512;
    k.hi512 = k.qhi + 512;

    // Batch i: statistics, then each row's output and stores.  The loads of
    // every batch of the pass were issued before the first store, so waiting
    // for a later batch's loads never waits for an earlier batch's stores.
    for (;;) {
#pragma unroll
        for (int i = 0; i < NB; ++i) {
            if (nr[i] <= 0) break;
            RowsStats<W, R> st;
            rows_stats<W, R>(a, k, xv[i], st);
            rows_output<W, R, CT>(a, k, s_gb, st, ra + R * i, nr[i], nd, lane, y32, yrs);
        }
        ra += NB * R;
        if (ra >= r1) break;
#pragma unroll
        for (int i = 0; i < NB; ++i) {
            nr[i] = (int)max<int64_t>(0, min<int64_t>(R, r1 - ra - R * i));
            load_rows<W, R, CT>(xv[i], xr, ra + R * i, nr[i], nd, lane, k.ok);
        }
    }
}

// Rows of fewer than 64 dwords (C < 256, C % 4 = 0, dword-aligned rows) whose
// per-lane sums of squares fit 32 bits.  L lanes own a row (R = 64 / L rows
// per pass, lane li holding dwords li, li + L, ...), and P passes form a
// batch.  The statistics of every pass are reduced over the row's L lanes;
// lane li < P of each row group keeps those of pass li, so that one square
// root and two divisions give the factors of P rows, which are broadcast back
// to the row's lanes pass by pass (ds_swizzle, no memory access).  The
// per-channel (gs, bs) pairs are read from LDS per element as in the
// row-batch kernel; a wavefront owns a contiguous run of rows in units of R.
template <int L>
__device__ __forceinline__ uint32_t seg_bcast(uint32_t v, int p) {
    static_assert(L >= 8 && L <= 32, "segments within a 32-lane swizzle group");
    // bitmask swizzle: lane' = (lane & and_mask) | or_mask within 32 lanes;
    // p is a constant once the callers' pass loops are unrolled
    constexpr int kAnd = 0x1F & ~(L - 1);
    int r;
    switch (p) {
        case 0: r = __builtin_amdgcn_ds_swizzle((int)v, kAnd | (0 << 5)); break;
        case 1: r = __builtin_amdgcn_ds_swizzle((int)v, kAnd | (1 << 5)); break;
        case 2: r = __builtin_amdgcn_ds_swizzle((int)v, kAnd | (2 << 5)); break;
        case 3: r = __builtin_amdgcn_ds_swizzle((int)v, kAnd | (3 << 5)); break;
        case 4: r = __builtin_amdgcn_ds_swizzle((int)v, kAnd | (4 << 5)); break;
        case 5: r = __builtin_amdgcn_ds_swizzle((int)v, kAnd | (5 << 5)); break;
        case 6: r = __builtin_amdgcn_ds_swizzle((int)v, kAnd | (6 << 5)); break;
        default: r = __builtin_amdgcn_ds_swizzle((int)v, kAnd | (7 << 5)); break;
    }
    return (uint32_t)r;
}

template <int L>
__device__ __forceinline__ double seg_bcast_f64(double v, int p) {
    const uint64_t u = (uint64_t)__double_as_longlong(v);
    const uint64_t lo = seg_bcast<L>((uint32_t)u, p), hi = seg_bcast<L>((uint32_t)(u >> 32), p);
    return __longlong_as_double((int64_t)((hi << 32) | lo));
}

// The lane's dwords of the batch's rows (pass p: row seg + p R of the batch;
// zeros for rows past nr and lanes past the row), as buffer loads that
// address past the input when not needed.  dw0 is the dword index of the
// lane's first dword in the batch's first row group (T C < 2^31 bytes).
// Stores the W packed dwords of a lane: one 4W-byte store (CT) or W dword
// stores L dwords apart.
template <int W, int L, bool CT>
__device__ __forceinline__ void store_seg(const uint32_t (&pk)[W], __amdgpu_buffer_rsrc_t yrs,
                                          int yoff, const bool (&ok)[W]) {
    if constexpr (CT) {
        if constexpr (W == 1) __builtin_amdgcn_raw_buffer_store_b32(pk[0], yrs, yoff, 0, 2);
        else if constexpr (W == 2) __builtin_amdgcn_raw_buffer_store_b64(u32x2_t{pk[0], pk[1]}, yrs, yoff, 0, 2);
        else if constexpr (W == 3)
            __builtin_amdgcn_raw_buffer_store_b96(u32x3_t{pk[0], pk[1], pk[2]}, yrs, yoff, 0, 2);
        else
            __builtin_amdgcn_raw_buffer_store_b128(u32x4_t{pk[0], pk[1], pk[2], pk[3]}, yrs, yoff, 0, 2);
    } else {
#pragma unroll
        for (int w = 0; w < W; ++w)
            if (ok[w]) __builtin_amdgcn_raw_buffer_store_b32(pk[w], yrs, yoff + 4 * L * w, 0, 2 /* nt */);
    }
}

template <int W, int L, int P, bool CT>
__device__ __forceinline__ void load_seg(uint32_t (&xv)[P][W], __amdgpu_buffer_rsrc_t xr,
                                         int dw0, int nr, int nd, int seg,
                                         const bool (&ok)[W]) {
    constexpr int R = 64 / L;
    if constexpr (CT) {
        // lane li holds dwords W li .. W li + W - 1 of its row (nd = L W)
#pragma unroll
        for (int p = 0; p < P; ++p) {
            const int off = p * R + seg < nr ? (dw0 + p * R * nd) * 4 : INT_MIN;
            if constexpr (W == 1) {
                xv[p][0] = __builtin_amdgcn_raw_buffer_load_b32(xr, off, 0, 0);
            } else if constexpr (W == 2) {
                const u32x2_t v = __builtin_amdgcn_raw_buffer_load_b64(xr, off, 0, 0);
                xv[p][0] = v[0]; xv[p][1] = v[1];
            } else if constexpr (W == 3) {
                const u32x3_t v = __builtin_amdgcn_raw_buffer_load_b96(xr, off, 0, 0);
                xv[p][0] = v[0]; xv[p][1] = v[1]; xv[p][2] = v[2];
            } else {
                const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(xr, off, 0, 0);
                xv[p][0] = v[0]; xv[p][1] = v[1]; xv[p][2] = v[2]; xv[p][3] = v[3];
            }
        }
        return;
    }
#pragma unroll
    for (int p = 0; p < P; ++p) {
#pragma unroll
        for (int w = 0; w < W; ++w) {
            const int off = (p * R + seg < nr && ok[w]) ? (dw0 + p * R * nd + L * w) * 4 : INT_MIN;
            xv[p][w] = __builtin_amdgcn_raw_buffer_load_b32(xr, off, 0, 0);
        }
    }
}

template <int W, int L, int P, int BLOCK, bool CT>
__global__ __launch_bounds__(BLOCK) void ln_seg_kernel(LnArgs a) {
    static_assert(P <= L && P <= 8, "lane li < P of a row group keeps pass li");
    constexpr int R = 64 / L;
    extern __shared__ double smem[];
    // all of it dynamic, so that the 16-byte entries stay 16-byte aligned
    double2* s_gb = reinterpret_cast<double2*>(smem);        // (gs, bs) at [b][dword]
    uint4* s_pk = reinterpret_cast<uint4*>(s_gb + a.C);      // per dword, as ln_rows_kernel
    const int nd = a.C >> 2;
    uint32_t* s_bnd = reinterpret_cast<uint32_t*>(s_pk + 2 * nd);   // bounds of |gs|
    const int lane = threadIdx.x & 63;
    const int seg = lane / L, li = lane % L;

    // contiguous run of units of R rows; wavefronts numbered across
    // workgroups first
    constexpr int kWaves = BLOCK / 64;
    const int64_t nw = (int64_t)gridDim.x * kWaves;
    const int64_t gw = (int64_t)__builtin_amdgcn_readfirstlane(threadIdx.x >> 6) * gridDim.x +
                       blockIdx.x;
    const int64_t units = (a.T + R - 1) / R;
    const int64_t ub = units / nw, urem = units % nw;
    const int64_t u0 = gw * ub + min(gw, urem);
    int64_t ra = u0 * R;
    const int64_t r1 = min<int64_t>(a.T, (u0 + ub + (gw < urem ? 1 : 0)) * R);
    // the whole input and output, a.T * a.C < 2^31 bytes (checked by the
    // launcher)
    const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
        (void*)a.x, (short)0, (int)(a.T * a.C), 0x00020000);
    const __amdgpu_buffer_rsrc_t yrs = __builtin_amdgcn_make_buffer_rsrc(
        (void*)a.y, (short)0, (int)(a.T * a.C), 0x00020000);
    RowsCtx<W> k;
#pragma unroll
    for (int w = 0; w < W; ++w) k.ok[w] = CT || li + L * w < nd;
    int dw0 = ((int)ra + seg) * nd + (CT ? W * li : li);

    // set-up as in ln_rows_kernel: one thread per dword (nd < 64), and the
    // bounds of |gs| over the whole row
    const int sdw = threadIdx.x;
    // LDS position of dword sdw (CT: dword W li + w at w L + li)
    const int spos = CT ? (sdw % W) * L + sdw / W : sdw;
    float sg[4], sb[4];
    int sa[4];
    if (sdw < nd) {
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            sg[b] = a.gamma[4 * sdw + b];
            sb[b] = a.beta[4 * sdw + b];
            sa[b] = a.alpha[4 * sdw + b];
        }
    }
    uint32_t xv[P][W];
    int nr = (int)max<int64_t>(0, min<int64_t>(P * R, r1 - ra));
    load_seg<W, L, P, CT>(xv, xr, dw0, nr, nd, seg, k.ok);

    const int u = a.zp_in + 128;
    uint32_t dhi = 0, dlo = 0x7FF00000u;
    if (sdw < nd) {
        uint32_t mulp[2] = {0, 0}, zmp[2] = {0, 0}, mulb = 0, m1p = 0;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            const double gs = (double)sg[b] / (double)a.s_out;
            s_gb[b * nd + spos] = double2{gs, (double)sb[b] / (double)a.s_out};
            const int sh = min(sa[b], a.K);
            const uint32_t zm = (uint32_t)(-u) << sh;
            mulb |= (1u << sh) << (8 * b);
            mulp[b >> 1] |= (1u << sh) << (16 * (b & 1));
            zmp[b >> 1] |= (zm & 0xFFFFu) << (16 * (b & 1));
            m1p += zm;
            const uint32_t h = (uint32_t)((uint64_t)__double_as_longlong(gs) >> 32) & 0x7FFFFFFFu;
            dhi = max(dhi, h);
            dlo = min(dlo, h);
        }
        s_pk[2 * spos] = uint4{mulp[0], mulp[1], zmp[0], zmp[1]};
        s_pk[2 * spos + 1] = uint4{mulb, m1p, 0u, 0u};
    }
    if (threadIdx.x < 64) {   // wave 0 holds every dword (nd < 64)
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            dhi = max(dhi, (uint32_t)__shfl_xor((int)dhi, off, 64));
            dlo = min(dlo, (uint32_t)__shfl_xor((int)dlo, off, 64));
        }
        if (threadIdx.x == 0) {
            s_bnd[0] = dhi;
            s_bnd[1] = dlo;
        }
    }
    __syncthreads();
    if (nr <= 0) return;

    k.m1init = 0;
#pragma unroll
    for (int w = 0; w < W; ++w) {
        const int dw = k.ok[w] ? li + L * w : 0;
        const uint4 p = s_pk[2 * dw];
        const uint4 q = s_pk[2 * dw + 1];
        k.mulp[2 * w] = k.ok[w] ? p.x : 0u;
        k.mulp[2 * w + 1] = k.ok[w] ? p.y : 0u;
        k.zmp[2 * w] = k.ok[w] ? p.z : 0u;
        k.zmp[2 * w + 1] = k.ok[w] ? p.w : 0u;
        k.mulb[w] = k.ok[w] ? q.x : 0u;
        k.m1init += k.ok[w] ? q.y : 0u;
    }
    // bounds of |gs| over the whole row from the high words (as in
    // ln_rows_kernel, here for every channel of the row)
    const uint32_t ghi = s_bnd[0], glo = s_bnd[1];
    k.gmaxl = __longlong_as_double((int64_t)(((uint64_t)ghi << 32) | 0xFFFFFFFFu));
    k.gminl = __longlong_as_double((int64_t)((uint64_t)glo << 32));
    k.zerol = glo == 0;
    k.qlo = -(1 << (a.bits - 1));
    k.qhi = (1 << (a.bits - 1)) - 1;
    k.hi_mask = ~((1u << (21 - a.bits)) - 1u);
    uint32_t m_add = ((uint32_t)(53 - a.bits) << 20) | 0x80000u;
    asm volatile("" : "+s"(m_add));
    k.m_add = m_add;
    k.amax = ldexp(1.0, a.bits);
    k.amin = ldexp(1.0, a.bits - 31);
    k.cadd = (double)a.zp_out + 512.5;
    k.lo512 = k.qlo + 512;
    k.hi512 = k.qhi + 512;

    for (;;) {
        // statistics of every pass; lane li keeps those of pass li
        uint32_t hp[P][2 * W];
        int cm1 = 0, clo = 0, chi = 0;
#pragma unroll
        for (int p = 0; p < P; ++p) {
            if (p * R >= nr) break;
            uint32_t m1 = k.m1init, m2 = 0;
#pragma unroll
            for (int w = 0; w < W; ++w) {
                const uint32_t xu = xv[p][w] ^ 0x80808080u;
                const uint32_t p0 = __builtin_amdgcn_perm(xu, xu, 0x0C010C00u);
                const uint32_t p1 = __builtin_amdgcn_perm(xu, xu, 0x0C030C02u);
                const short2_t h0 = __builtin_bit_cast(short2_t, p0) * __builtin_bit_cast(short2_t, k.mulp[2 * w]) +
                                    __builtin_bit_cast(short2_t, k.zmp[2 * w]);
                const short2_t h1 = __builtin_bit_cast(short2_t, p1) * __builtin_bit_cast(short2_t, k.mulp[2 * w + 1]) +
                                    __builtin_bit_cast(short2_t, k.zmp[2 * w + 1]);
                m1 = __builtin_amdgcn_udot4(xu, k.mulb[w], m1, false);
                m2 = (uint32_t)__builtin_amdgcn_sdot2(h0, h0, (int)m2, false);
                m2 = (uint32_t)__builtin_amdgcn_sdot2(h1, h1, (int)m2, false);
                hp[p][2 * w] = __builtin_bit_cast(uint32_t, h0);
                hp[p][2 * w + 1] = __builtin_bit_cast(uint32_t, h1);
            }
            // per-lane m2 < 2^32: its 16-bit halves are summed separately
            const int s1 = dpp_seg_sum((int)m1, L);
            const int slo = dpp_seg_sum((int)(m2 & 0xFFFFu), L);
            const int shi = dpp_seg_sum((int)(m2 >> 16), L);
            cm1 = li == p ? s1 : cm1;
            clo = li == p ? slo : clo;
            chi = li == p ? shi : chi;
        }
        double r, m;
        row_factors((int64_t)cm1, ((int64_t)chi << 16) + clo, a.C, r, m);
        const uint32_t fast = (r > 0.0 && !k.zerol && k.gmaxl * r < k.amax && k.gminl * r >= k.amin) ? 1u : 0u;

#pragma unroll
        for (int p = 0; p < P; ++p) {
            if (p * R >= nr) break;
            const double rp = seg_bcast_f64<L>(r, p);
            const double mp = seg_bcast_f64<L>(m, p);
            const bool fp = seg_bcast<L>(fast, p) != 0u;
            const int j = p * R + seg;
            const int yoff = (dw0 + p * R * nd) * 4;   // the lane's first dword of the row
            if (j < nr && fp) {
                uint32_t packs[W];
#pragma unroll
                for (int w = 0; w < W; ++w) {
                    int q[4];
#pragma unroll
                    for (int b = 0; b < 4; ++b) {
                        const uint32_t hw = hp[p][2 * w + (b >> 1)];
                        const int xh = (b & 1) ? (int)hw >> 16 : (int)(int16_t)(hw & 0xFFFFu);
                        const double2 gb = s_gb[b * nd + (k.ok[w] ? li + L * w : 0)];
                        const double A = gb.x * rp;
                        const double B = gb.y - gb.x * mp;
                        q[b] = ln_requant_rows(A, B, xh, k.hi_mask, k.m_add, k.cadd, k.lo512, k.hi512);
                    }
                    const uint32_t lo = __builtin_amdgcn_perm((uint32_t)q[1], (uint32_t)q[0], 0x0C0C0400u);
                    const uint32_t hi = __builtin_amdgcn_perm((uint32_t)q[3], (uint32_t)q[2], 0x0C0C0400u);
                    packs[w] = __builtin_amdgcn_perm(hi, lo, 0x05040100u);
                    if (!CT && k.ok[w])
                        __builtin_amdgcn_raw_buffer_store_b32(packs[w], yrs, yoff + 4 * L * w, 0, 2 /* nt */);
                    __builtin_amdgcn_sched_barrier(0);
                }
                if (CT) store_seg<W, L, true>(packs, yrs, yoff, k.ok);
            } else if (j < nr) {
                uint32_t packs[W];
#pragma unroll
                for (int w = 0; w < W; ++w) {
                    uint32_t pack = 0;
#pragma unroll
                    for (int b = 0; b < 4; ++b) {
                        const uint32_t hw = hp[p][2 * w + (b >> 1)];
                        const int xh = (b & 1) ? (int)hw >> 16 : (int)(int16_t)(hw & 0xFFFFu);
                        const double2 gb = s_gb[b * nd + (k.ok[w] ? li + L * w : 0)];
                        const double A = gb.x * rp;
                        const double B = gb.y - gb.x * mp;
                        const int q = ln_requant(A, B, xh, a.bits, a.zp_out, k.qlo, k.qhi);
                        pack |= ((uint32_t)q & 0xFFu) << (8 * b);
                    }
                    packs[w] = pack;
                }
                store_seg<W, L, CT>(packs, yrs, yoff, k.ok);
            }
        }
        ra += P * R;
        dw0 += P * R * nd;
        if (ra >= r1) break;
        nr = (int)max<int64_t>(0, min<int64_t>(P * R, r1 - ra));
        load_seg<W, L, P, CT>(xv, xr, dw0, nr, nd, seg, k.ok);
    }
}

template <int W, int R, int NB, bool SPREAD, int BLOCK>
hipError_t launch_rows_rb(const LnArgs& a, int wpc, hipStream_t stream) {
    // one pass of NB batches of R rows per wavefront where the rows allow it
    // (SPREAD: one batch of R rows per wavefront, the later batches of a pass
    // holding the remainder), at most wpc wavefronts per CU
    constexpr int kWaves = BLOCK / 64;
    const int64_t want = SPREAD ? (a.T + R - 1) / R : (a.T + NB * R - 1) / (NB * R);
    const int64_t waves = std::max<int64_t>(1, std::min<int64_t>(want, 256 * (int64_t)wpc));
    const int64_t blocks = (waves + kWaves - 1) / kWaves;
    const size_t lds = (size_t)a.C * 2 * sizeof(double) + (size_t)(a.C / 4) * 2 * sizeof(uint4);
    if (a.C == 256 * W)
        launch_kernel(ln_rows_kernel<W, R, BLOCK, NB, true>, dim3((unsigned)blocks), dim3(BLOCK),
                      lds, stream, a);
    else
        launch_kernel(ln_rows_kernel<W, R, BLOCK, NB, false>, dim3((unsigned)blocks), dim3(BLOCK),
                      lds, stream, a);
    return hipGetLastError();
}

// Twelve wavefronts per CU.  Where the rows fill all of them, one workgroup of
// twelve wavefronts per CU: the per-channel set-up (binary64 divisions, packed
// constants) then runs once per CU instead of once per four wavefronts.  Rows
// come in batches of four where there are at least four per wavefront, else in
// batches of two (two per pass, the second holding the remainder), which gives
// more wavefronts.  Measured on one MI355X, kernel events, all bit-identical:
//   ViT-B/16 (12608 x 768): 11.3 us with 256-thread workgroups and each
//   batch's stores held back until the next batch's loads had arrived; 11.0 us
//   with each row stored as soon as it is computed; 10.4 us with one
//   workgroup per CU (two-row batches 10.7 us; 512-thread workgroups 11.7-12.2
//   us; 16 wavefronts per CU 11.7-16.0 us).
//   ViT-L/16 (9232 x 1024): 12.5 us before; four-row batches 12.2 us
//   (2308 wavefronts); two-row batches 11.2 us with 256-thread workgroups and
//   10.5 us with one workgroup per CU.
//   DeiT-S (1576 x 384): 5.4 us before; two-row batches 4.1 us with 256-thread
//   workgroups, 5.2 us with 768 (66 CUs busy instead of 197).
// Three or more batches per pass, single-row batches, or eight or sixteen
// wavefronts per CU were slower on every shape.  The kernel stays bound by
// its vector-ALU issue (the binary64 output).
template <int W>
hipError_t launch_rows(const LnArgs& a, hipStream_t stream) {
    constexpr int kWpc = 12;
    const int64_t full = 256 * (int64_t)kWpc;
    if ((a.T + 3) / 4 >= full) return launch_rows_rb<W, 4, 1, false, 64 * kWpc>(a, kWpc, stream);
    if ((a.T + 1) / 2 >= full) return launch_rows_rb<W, 2, 2, true, 64 * kWpc>(a, kWpc, stream);
    return launch_rows_rb<W, 2, 2, true, 256>(a, kWpc, stream);
}

template <int W, int L, int P, int BLOCK>
hipError_t launch_seg_b(const LnArgs& a, int wpc, hipStream_t stream) {
    constexpr int kWaves = BLOCK / 64;
    constexpr int R = 64 / L;
    const int64_t want = (a.T + R * P - 1) / (R * P);
    const int64_t waves = std::max<int64_t>(1, std::min<int64_t>(want, 256 * (int64_t)wpc));
    const int64_t blocks = (waves + kWaves - 1) / kWaves;
    const size_t lds =
        (size_t)a.C * 2 * sizeof(double) + (size_t)(a.C / 4) * 2 * sizeof(uint4) + sizeof(uint4);
    if (a.C == 4 * L * W)
        launch_kernel(ln_seg_kernel<W, L, P, BLOCK, true>, dim3((unsigned)blocks), dim3(BLOCK), lds,
                      stream, a);
    else
        launch_kernel(ln_seg_kernel<W, L, P, BLOCK, false>, dim3((unsigned)blocks), dim3(BLOCK), lds,
                      stream, a);
    return hipGetLastError();
}

// Twelve wavefronts per CU.  Where batches of four passes fill them all (or
// else of two), one workgroup per CU; fewer rows take single passes, which
// gives the most wavefronts.  Measured on one MI355X, kernel events, all
// bit-identical:
//   Swin-S (100352 x 96, L = 8): 15.3 us with the earlier kernel (factors of
//   every pass computed on their own, gs and bs held in registers); batches
//   of 1, 2, 4 or 8 passes 13.8, 11.8, 11.4 and 14.3 us with one workgroup
//   per CU (256-thread workgroups 0.3-0.8 us slower; 16 wavefronts per CU
//   slower still).  The static LDS of an earlier form left the 16-byte
//   (gs, bs) entries 8-byte aligned: 21-22 us.
//   DeiT-Ti (197 x 192, L = 16): 4.4 us before; 1, 2, 4 or 8 passes 4.0,
//   4.2, 5.4 and 7.8 us.
template <int W, int L>
hipError_t launch_seg_l(const LnArgs& a, hipStream_t stream) {
    constexpr int kWpc = 12;
    constexpr int R = 64 / L;
    const int64_t full = 256 * (int64_t)kWpc;
    if ((a.T + 4 * R - 1) / (4 * R) >= full) return launch_seg_b<W, L, 4, 64 * kWpc>(a, kWpc, stream);
    if ((a.T + 2 * R - 1) / (2 * R) >= full) return launch_seg_b<W, L, 2, 64 * kWpc>(a, kWpc, stream);
    return launch_seg_b<W, L, 1, 256>(a, kWpc, stream);
}

template <int W>
hipError_t launch_seg(const LnArgs& a, int lshift, hipStream_t stream) {
    switch (lshift) {
        case 3: return launch_seg_l<W, 8>(a, stream);
        case 4: return launch_seg_l<W, 16>(a, stream);
        default: return launch_seg_l<W, 32>(a, stream);
    }
}

template <int W>
hipError_t launch_fast(const LnArgs& a, int lshift, bool wide, hipStream_t stream) {
    const int R = 64 >> lshift;
    const int64_t waves = (a.T + R - 1) / R;
    const int64_t blocks = std::min<int64_t>((waves + 3) / 4, 1024);
    const size_t lds = (size_t)a.C * (2 * sizeof(double) + sizeof(int));
    if (wide)
        launch_kernel(ln_fast_kernel<W, true>, dim3((unsigned)blocks), dim3(kBlock), lds,
                           stream, a, lshift);
    else
        launch_kernel(ln_fast_kernel<W, false>, dim3((unsigned)blocks), dim3(kBlock), lds,
                           stream, a, lshift);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_ptf_layernorm(const LnArgs& a, hipStream_t stream) {
    const bool aligned = ((reinterpret_cast<uintptr_t>(a.x) | reinterpret_cast<uintptr_t>(a.y)) & 3) == 0;
    // Lanes per row L and dwords per lane W: least padding, then the most
    // lanes per row (fewest registers, highest occupancy).
    const int nd = a.C / 4;
    const bool narrow = (double)a.C * 65025.0 * (double)(1 << (2 * a.K)) < 4294967296.0;
    // Row-batch kernel for 256 <= C <= 1024 (up to 4 dwords per lane without
    // spills) when the sums of squares fit 32 bits.
    if (aligned && a.C % 4 == 0 && nd >= 64 && nd <= 256 && narrow &&
        a.T * (int64_t)a.C < ((int64_t)1 << 31)) {
        switch ((nd + 63) / 64) {
            case 1: return launch_rows<1>(a, stream);
            case 2: return launch_rows<2>(a, stream);
            case 3: return launch_rows<3>(a, stream);
            default: return launch_rows<4>(a, stream);
        }
    }
    int best_l = -1, best_w = 0, best_waste = 1 << 30;
    if (aligned && a.C % 4 == 0) {
        for (int l = 6; l >= 0; --l) {
            const int L = 1 << l;
            const int W = (a.C / 4 + L - 1) / L;
            if (W > 8) continue;
            const int waste = 4 * W * L - a.C;
            if (waste < best_waste) {
                best_waste = waste;
                best_l = l;
                best_w = W;
            }
        }
    }
    if (best_l < 0) {
        const int64_t blocks = std::min<int64_t>((a.T + 3) / 4, 2048);
        launch_kernel(ln_generic_kernel, dim3((unsigned)blocks), dim3(kBlock), 0, stream, a);
        return hipGetLastError();
    }
    // Per-lane sums of squares: 4W values of at most (255 * 2^K)^2 each.
    const bool wide = (double)(4 * best_w) * 65025.0 * (double)(1 << (2 * a.K)) >= 2147483647.0;
    // The choice above gives odd W wherever L < 64: an even W ties with twice
    // the lanes and half the dwords, which the scan (most lanes first) keeps.
    if (!wide && best_l >= 3 && best_l <= 5 && (best_w == 1 || best_w == 3) &&
        a.T * (int64_t)a.C < ((int64_t)1 << 31))
        return best_w == 1 ? launch_seg<1>(a, best_l, stream) : launch_seg<3>(a, best_l, stream);
    switch (best_w) {
        case 1: return launch_fast<1>(a, best_l, wide, stream);
        case 2: return launch_fast<2>(a, best_l, wide, stream);
        case 3: return launch_fast<3>(a, best_l, wide, stream);
        case 4: return launch_fast<4>(a, best_l, wide, stream);
        case 5: return launch_fast<5>(a, best_l, wide, stream);
        case 6: return launch_fast<6>(a, best_l, wide, stream);
        case 7: return launch_fast<7>(a, best_l, wide, stream);
        default: return launch_fast<8>(a, best_l, wide, stream);
    }
}

}  // namespace fqvit
