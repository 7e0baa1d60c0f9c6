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
// Layout: one row is handled by L lanes (L a power of two <= 64, 64/L rows per
// wavefront), each lane owning W 4-channel dwords of the row, so that the
// loads are coalesced dwords and the row statistics are a segmented
// shuffle reduction.  Per-channel gs, bs and the clamped shift are computed
// once per workgroup into LDS and then held in registers; waves stride over
// rows.
#include "fqvit_internal.h"

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

// Output of one element when A = gs r is known to lie in [2^(b-31), 2^b): then
// N1 = b - 1 - floor(log2 |A|) needs no clamp and sign(A) N2 / 2^N1 is A with
// its significand cut to b bits, a mask on the high word (b <= 8 keeps the
// low word zero).  rint(B 2^N1) 2^-N1 is B rounded to the grid of that last
// bit, 2^(E - b + 1) with E the exponent of A, ties to even: adding and
// subtracting M = 1.5 2^(E - b + 53) does exactly that while |B| < 2^(E - b + 52);
// larger B (and the oracle's clamp of B 2^N1 at 2^62) saturate the output
// either way, since |A X^| < 2^(E + 12).  Same result as ln_requant.
// m_add = (53 - b) << 20 | 0x80000 builds M's high word from A's exponent
// field; dlo, dhi: the output bounds minus zp_out.
__device__ __forceinline__ int ln_requant_fast(double A, double B, int xh, uint32_t hi_mask,
                                               uint32_t m_add, int zp_out, double dlo,
                                               double dhi) {
    const uint32_t hiA = (uint32_t)((uint64_t)__double_as_longlong(A) >> 32);
    const double At = __longlong_as_double((int64_t)((uint64_t)(hiA & hi_mask) << 32));
    const double M = __longlong_as_double((int64_t)((uint64_t)((hiA & 0x7FF00000u) + m_add) << 32));
    const double Bg = (B + M) - M;
    const double val = fma(At, (double)xh, Bg + 0.5);
    return (int)floor(fmin(fmax(val, dlo), dhi)) + zp_out;
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

    const int qlo = -(1 << (a.bits - 1));
    const int qhi = (1 << (a.bits - 1)) - 1;
    const uint32_t hi_mask = ~((1u << (21 - a.bits)) - 1u);   // keep sign, exponent, b-1 bits
    const uint32_t m_add = ((uint32_t)(53 - a.bits) << 20) | 0x80000u;
    const double amax = ldexp(1.0, a.bits), amin = ldexp(1.0, a.bits - 31);
    const double dlo = (double)(qlo - a.zp_out), dhi = (double)(qhi - a.zp_out);
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
        int m1 = 0;
        uint32_t m2 = 0;
        int64_t m2w = 0;
#pragma unroll
        for (int w = 0; w < W; ++w) {
#pragma unroll
            for (int b = 0; b < 4; ++b) {
                const int x = (int)(int8_t)(xv[w] >> (8 * b));
                const int h = __mul24(x - a.zp_in, mul[4 * w + b]);   // 0 past C
                xh[4 * w + b] = h;
                m1 += h;
                if (WIDE) m2w += (int64_t)h * h;
                else m2 += (uint32_t)__mul24(h, h);
            }
        }
        int64_t M1, M2;
        if (WIDE) {
            M1 = seg_sum<int>(m1, L);
            M2 = seg_sum<int64_t>(m2w, L);
        } else {
            // per-lane m2 < 2^31: sum its 16-bit halves separately in 32 bits
            M1 = dpp_seg_sum(m1, L);
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
                uint32_t pack = 0;
#pragma unroll
                for (int b = 0; b < 4; ++b) {
                    const int k = 4 * w + b;
                    const double A = gs[k] * r;
                    const double B = bs[k] - gs[k] * m;
                    const int q = ln_requant_fast(A, B, xh[k], hi_mask, m_add, a.zp_out, dlo, dhi);
                    pack |= ((uint32_t)q & 0xFFu) << (8 * b);
                }
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
