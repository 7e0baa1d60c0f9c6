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

// Fast path: C % 4 == 0, dword-aligned rows, W dwords per lane (W <= 8).
// WIDE selects 64-bit per-lane sums of squares (K >= 6).
template <int W, bool WIDE>
__global__ __launch_bounds__(kBlock) void ln_fast_kernel(LnArgs a, int lshift) {
    extern __shared__ double smem[];
    double* s_gs = smem;
    double* s_bs = smem + a.C;
    int* s_mul = reinterpret_cast<int*>(smem + 2 * a.C);
    for (int c = threadIdx.x; c < a.C; c += blockDim.x) {
        s_gs[c] = (double)a.gamma[c] / (double)a.s_out;
        s_bs[c] = (double)a.beta[c] / (double)a.s_out;
        s_mul[c] = 1 << min((int)a.alpha[c], a.K);
    }
    __syncthreads();

    const int lane = threadIdx.x & 63;
    const int L = 1 << lshift;
    const int seg = lane >> lshift;
    const int li = lane & (L - 1);
    const int R = 64 >> lshift;
    const int nd = a.C >> 2;

    double gs[4 * W], bs[4 * W];
    int mul[4 * W];
    bool ok[W];
#pragma unroll
    for (int w = 0; w < W; ++w) {
        const int dw = li + (w << lshift);
        ok[w] = dw < nd;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            const int c = ok[w] ? 4 * dw + b : 0;
            gs[4 * w + b] = s_gs[c];
            bs[4 * w + b] = s_bs[c];
            mul[4 * w + b] = ok[w] ? s_mul[c] : 0;
        }
    }

    const int qlo = -(1 << (a.bits - 1));
    const int qhi = (1 << (a.bits - 1)) - 1;
    const int64_t gw = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    const int64_t nw = ((int64_t)gridDim.x * blockDim.x) >> 6;

    for (int64_t r0 = gw * R; r0 < a.T; r0 += nw * R) {
        const int64_t row = r0 + seg;
        const bool rok = row < a.T;
        const int64_t rr = rok ? row : 0;
        const uint32_t* xr = reinterpret_cast<const uint32_t*>(a.x + rr * a.C);
        uint32_t xv[W];
#pragma unroll
        for (int w = 0; w < W; ++w)
            xv[w] = ok[w] ? __builtin_nontemporal_load(xr + li + (w << lshift)) : 0u;

        int xh[4 * W];
        int m1 = 0;
        int m2 = 0;
        int64_t m2w = 0;
#pragma unroll
        for (int w = 0; w < W; ++w) {
#pragma unroll
            for (int b = 0; b < 4; ++b) {
                const int x = (int)(int8_t)(xv[w] >> (8 * b));
                const int h = (x - a.zp_in) * mul[4 * w + b];   // 0 for channels past C
                xh[4 * w + b] = h;
                m1 += h;
                if (WIDE) m2w += (int64_t)h * h;
                else m2 += h * h;
            }
        }
        const int64_t M1 = seg_sum<int>(m1, L);
        const int64_t M2 = WIDE ? seg_sum<int64_t>(m2w, L) : seg_sum<int64_t>((int64_t)m2, L);
        double r, m;
        row_factors(M1, M2, a.C, r, m);

        uint32_t* yr = reinterpret_cast<uint32_t*>(a.y + rr * a.C);
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
        hipLaunchKernelGGL((ln_fast_kernel<W, true>), dim3((unsigned)blocks), dim3(kBlock), lds,
                           stream, a, lshift);
    else
        hipLaunchKernelGGL((ln_fast_kernel<W, false>), dim3((unsigned)blocks), dim3(kBlock), lds,
                           stream, a, lshift);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_ptf_layernorm(const LnArgs& a, hipStream_t stream) {
    const bool aligned = ((reinterpret_cast<uintptr_t>(a.x) | reinterpret_cast<uintptr_t>(a.y)) & 3) == 0;
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
        hipLaunchKernelGGL(ln_generic_kernel, dim3((unsigned)blocks), dim3(kBlock), 0, stream, a);
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
