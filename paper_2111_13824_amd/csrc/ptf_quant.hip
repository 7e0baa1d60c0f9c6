// PTF calibration and quantization (Sec. 3.2, eq. 8-11) and the dyadic
// requantization of an int32 accumulator (the integer form of Supplement A.1)
// for gfx950.
//
// Calibration runs four kernels:
//   1. minmax_partial  per-workgroup minimum and maximum of x;
//   2. calib_params    the layer-wise scale s = (max - min) / (2^b - 1) / 2^K
//                      and zero point zp = clip(rint(-min / (2^K s)), 0, 2^b - 1)
//                      in binary64 (eq. 9, 10), each operation rounded once;
//   3. alpha_partial   for every channel c and block of 64 consecutive rows
//                      the squared errors of the K + 1 candidate grids summed
//                      in row order (eq. 11 with its zero point and clip);
//   4. alpha_select    per channel and alpha, the block sums added in block
//                      order, then per channel the argmin over alpha (the
//                      smallest on ties).
// Steps 3 and 4 fix the summation order, so the argmin is a pure function of
// x.  Against the exact argmin of eq. (11) (an exact sum of exact squares) the
// binary64 terms and sums can only swap candidates whose exact errors differ
// by less than the sum of their rounding bounds, (T + 8) 2^-53 times
// sum_t (|x| + 2 |deq|)^2 each.  x / (2^alpha s) is computed as ldexp(x / s,
// -alpha): scaling by a power of two commutes with the rounding of the
// quotient, which never leaves the normal range for binary32 inputs.
#include <cmath>
#include <mutex>

#include "fqvit.h"
#include "fqvit_launch.h"

namespace fqvit {
namespace {

constexpr int kBlock = 256;

typedef float vf4 __attribute__((ext_vector_type(4)));
typedef int vi4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float wave_min(float v) {
    for (int off = 32; off >= 1; off >>= 1) v = fminf(v, __shfl_xor(v, off, 64));
    return v;
}

__device__ __forceinline__ float wave_max(float v) {
    for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
    return v;
}

// part[2 b], part[2 b + 1] = minimum and maximum of workgroup b's elements.
__global__ __launch_bounds__(kBlock) void minmax_partial_kernel(const float* x, int64_t n,
                                                                int vec4, float* part) {
    float mn = INFINITY, mx = -INFINITY;
    const int64_t tid = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    if (vec4) {
        const vf4* x4 = reinterpret_cast<const vf4*>(x);
        for (int64_t i = tid; i < n / 4; i += stride) {
            const vf4 v = __builtin_nontemporal_load(x4 + i);
            mn = fminf(fminf(mn, v.x), fminf(v.y, fminf(v.z, v.w)));
            mx = fmaxf(fmaxf(mx, v.x), fmaxf(v.y, fmaxf(v.z, v.w)));
        }
        for (int64_t i = (n / 4) * 4 + tid; i < n; i += stride) {
            mn = fminf(mn, x[i]);
            mx = fmaxf(mx, x[i]);
        }
    } else {
        for (int64_t i = tid; i < n; i += stride) {
            mn = fminf(mn, x[i]);
            mx = fmaxf(mx, x[i]);
        }
    }
    __shared__ float s_mn[kBlock / 64], s_mx[kBlock / 64];
    mn = wave_min(mn);
    mx = wave_max(mx);
    if ((threadIdx.x & 63) == 0) {
        s_mn[threadIdx.x >> 6] = mn;
        s_mx[threadIdx.x >> 6] = mx;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < kBlock / 64; ++w) {
            mn = fminf(mn, s_mn[w]);
            mx = fmaxf(mx, s_mx[w]);
        }
        part[2 * blockIdx.x] = mn;
        part[2 * blockIdx.x + 1] = mx;
    }
}

// The overall minimum and maximum from the min/max partials (every thread of
// the workgroup gets them), then s and zp (container form) as in eq. (9),
// (10).  A tensor with max == min (or a non-finite range) gets s = 0 and the
// zero point 0 of the paper's grid.
__device__ void calib_params(const float* part, int nparts, int bits, int K, double& s_out,
                             int32_t& zp_out) {
    float mn = INFINITY, mx = -INFINITY;
    for (int i = threadIdx.x; i < nparts; i += kBlock) {
        mn = fminf(mn, part[2 * i]);
        mx = fmaxf(mx, part[2 * i + 1]);
    }
    __shared__ float s_mn[kBlock / 64], s_mx[kBlock / 64];
    mn = wave_min(mn);
    mx = wave_max(mx);
    if ((threadIdx.x & 63) == 0) {
        s_mn[threadIdx.x >> 6] = mn;
        s_mx[threadIdx.x >> 6] = mx;
    }
    __syncthreads();
    mn = s_mn[0];
    mx = s_mx[0];
    for (int w = 1; w < kBlock / 64; ++w) {
        mn = fminf(mn, s_mn[w]);
        mx = fmaxf(mx, s_mx[w]);
    }
    const double levels = (double)((1 << bits) - 1);
    const double two_K = ldexp(1.0, K);
    const double s = ((double)mx - (double)mn) / levels / two_K;
    const int half = 1 << (bits - 1);
    if (!(s > 0.0) || !isfinite(s)) {
        s_out = 0.0;
        zp_out = -half;
        return;
    }
    const double z = fmin(fmax(rint(-(double)mn / (two_K * s)), 0.0), levels);
    s_out = s;
    zp_out = (int32_t)z - half;
}

// One workgroup: s and zp from the min/max partials, stored for the kernels
// that follow.
__global__ __launch_bounds__(kBlock) void calib_params_kernel(const float* mm, int nparts, int bits,
                                                              int K, double* s_store,
                                                              int32_t* zp_store) {
    double s;
    int32_t zpc;
    calib_params(mm, nparts, bits, K, s, zpc);
    if (threadIdx.x == 0) {
        *s_store = s;
        *zp_store = zpc;
    }
}

// Workgroup (cx, k): channels cx*64 .. cx*64 + 63 (one per lane) and the
// rows of block k, taken in two halves of 32 rows.  For each half, every
// wavefront loads 8 of its rows and forms x / s (one correctly rounded
// division per element); x and the quotient go to LDS.  Wavefront w takes the
// candidates alpha = w, w + 4, ...: it runs down the rows in order and adds
// the terms (x - deq_a(x))^2 one at a time, carrying its sums from the first
// half to the second, part[(a nb + k) C + c] = ((0 + term_0) + term_1) + ...
// The row loads are issued before s and zp are read.
constexpr int kHalfRows = kPtfErrBlock / 2;
constexpr int kRowsPerWave = kHalfRows / (kBlock / 64);
constexpr int kAlphaPerWave = 2;    // candidates per wavefront (K <= 7)

template <int K>
__global__ __launch_bounds__(kBlock) void alpha_partial_kernel(const float* x, int64_t T, int C,
                                                               int bits, const double* s_ptr,
                                                               const int32_t* zp_ptr, int64_t nb,
                                                               double* part) {
    static_assert(K + 1 <= kAlphaPerWave * (kBlock / 64), "candidates per wavefront");
    __shared__ float xs[kHalfRows][64];            // 8 KB
    __shared__ double qs[kHalfRows][64];           // 16 KB: x / s
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int c = blockIdx.x * 64 + lane;
    const int64_t k = blockIdx.y;
    const int64_t t0 = k * kPtfErrBlock;
    const int nt = (int)min<int64_t>(kPtfErrBlock, T - t0);   // rows in this block
    const int r0 = wave * kRowsPerWave;

    float xv[2][kRowsPerWave];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
#pragma unroll
        for (int i = 0; i < kRowsPerWave; ++i) {
            const int r = h * kHalfRows + r0 + i;
            xv[h][i] = (c < C && r < nt) ? x[(t0 + r) * C + c] : 0.0f;
        }
    }
    const double s = *s_ptr;
    const int32_t zpc = *zp_ptr;
    if (!(s > 0.0)) return;                        // uniform over the grid
    const double zp = (double)(zpc + (1 << (bits - 1)));
    const double lo = -zp, hi = (double)((1 << bits) - 1) - zp;

    double acc[kAlphaPerWave];
#pragma unroll
    for (int j = 0; j < kAlphaPerWave; ++j) acc[j] = 0.0;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        if (h) __syncthreads();                    // the first half is consumed
#pragma unroll
        for (int i = 0; i < kRowsPerWave; ++i) {
            xs[r0 + i][lane] = xv[h][i];
            qs[r0 + i][lane] = (double)xv[h][i] / s;
        }
        __syncthreads();
        const int nh = min(kHalfRows, nt - h * kHalfRows);
#pragma unroll
        for (int j = 0; j < kAlphaPerWave; ++j) {
            const int a = wave + j * (kBlock / 64);
            if (a > K) break;
            const double step = ldexp(s, a);
            double sum = acc[j];
            // clamp(rint(.) + zp, 0, levels) - zp as one clamp of the integer
            // rint(.) to [-zp, levels - zp]: the same value, all exact
#pragma unroll 8
            for (int r = 0; r < nh; ++r) {
                const double qz = fmin(fmax(rint(ldexp(qs[r][lane], -a)), lo), hi);
                const double deq = qz * step;
                const double e = (double)xs[r][lane] - deq;
                const double term = e * e;
                sum = sum + term;
            }
            acc[j] = sum;
        }
    }
#pragma unroll
    for (int j = 0; j < kAlphaPerWave; ++j) {
        const int a = wave + j * (kBlock / 64);
        if (a <= K && c < C) part[((int64_t)a * nb + k) * C + c] = acc[j];
    }
}

// Error sums and the argmin of eq. 11 in one launch.  Workgroup g owns the
// channels g*cb .. g*cb + cb - 1 with cb = kSelChains / (K + 1), i.e. cb (K + 1)
// chains (channel, alpha).  The block sums of each chain are staged in LDS, up
// to kSelRows blocks per pass (loaded by the whole workgroup), and the chain's
// lane of wavefront 0 adds them in block order:
//     err(c, a) = ((0 + part_0) + part_1) + ...
// Then one lane per channel takes the argmin over alpha, ties to the smallest.
constexpr int kSelChains = 16;
constexpr int kSelRows = 256;    // 32 KB of LDS per pass
constexpr int kSelPerThread = kSelRows * kSelChains / kBlock;

__global__ __launch_bounds__(kBlock) void alpha_select_kernel(const double* part, int C, int K,
                                                              int64_t nb, const double* s_ptr,
                                                              uint8_t* alpha) {
    __shared__ double tile[kSelRows * kSelChains];
    __shared__ double err[kSelChains];
    const int cb = kSelChains / (K + 1);
    const int nch = cb * (K + 1);
    const int c0 = blockIdx.x * cb;
    const int t = threadIdx.x;
    if (!(*s_ptr > 0.0)) {
        if (t < cb && c0 + t < C) alpha[c0 + t] = 0;
        return;
    }
    double acc = 0.0;
    for (int64_t k0 = 0; k0 < nb; k0 += kSelRows) {
        const int nk = (int)min<int64_t>(kSelRows, nb - k0);
        // all of this thread's loads first, then the LDS stores
        double v[kSelPerThread];
#pragma unroll
        for (int i = 0; i < kSelPerThread; ++i) {
            const int idx = t + i * kBlock;
            const int row = idx / kSelChains, ch = idx - row * kSelChains;
            const int a = ch / cb, c = c0 + ch - a * cb;
            v[i] = (row < nk && ch < nch && c < C) ? part[((int64_t)a * nb + k0 + row) * C + c] : 0.0;
        }
        __syncthreads();   // the previous pass's sums have read the tile
#pragma unroll
        for (int i = 0; i < kSelPerThread; ++i) tile[t + i * kBlock] = v[i];
        __syncthreads();
        if (t < nch)
            for (int r = 0; r < nk; ++r) acc = acc + tile[r * kSelChains + t];
    }
    if (t < nch) err[t] = acc;
    __syncthreads();
    if (t < cb && c0 + t < C) {
        int best = 0;
        double best_err = INFINITY;
        for (int a = 0; a <= K; ++a) {
            const double e = err[a * cb + t];
            if (e < best_err) {
                best_err = e;
                best = a;
            }
        }
        alpha[c0 + t] = (uint8_t)best;
    }
}

// X_Q = clip(rint(x / (2^alpha_c s)) + zp, 0, 2^b - 1) (eq. 8), stored in the
// int8 container.  A thread covers four consecutive channels of one row.
// s <= 0 (a degenerate calibration) stores the zero point.
__device__ __forceinline__ int ptf_q(float x, double s, double zp, double levels, int a) {
    const double q = fmin(fmax(rint(ldexp((double)x / s, -a)) + zp, 0.0), levels);
    return (int)q;
}

// Thread (quad, row slot): channels 4 quad .. 4 quad + 3 with quad =
// 64 blockIdx.x + lane, and kQuantRows rows spaced 4 gridDim.y apart from
// 4 blockIdx.y + wavefront, all loaded before any is converted; a wavefront's
// 64 quads are 1 KB of contiguous input.  The channels' alphas are read once
// per thread.
constexpr int kQuantRows = 4;

__global__ __launch_bounds__(kBlock) void quantize_kernel(const float* x, int64_t T, int C,
                                                          const double* s_ptr,
                                                          const int32_t* zp_ptr,
                                                          const uint8_t* alpha, int bits,
                                                          int vec4, int8_t* y) {
    const double s = *s_ptr;
    const int half = 1 << (bits - 1);
    const int zpc = *zp_ptr;
    const double zp = (double)(zpc + half);
    const double levels = (double)((1 << bits) - 1);
    const int cq = (C + 3) >> 2;
    const int quad = blockIdx.x * 64 + (threadIdx.x & 63);
    if (quad >= cq) return;
    const int c0 = quad * 4;
    int al[4];
#pragma unroll
    for (int b = 0; b < 4; ++b) al[b] = c0 + b < C ? alpha[c0 + b] : 0;
    const int64_t step = (int64_t)gridDim.y * 4;
    for (int64_t t0 = (int64_t)blockIdx.y * 4 + (threadIdx.x >> 6); t0 < T;
         t0 += step * kQuantRows) {
        if (vec4) {
            vf4 v[kQuantRows];
#pragma unroll
            for (int j = 0; j < kQuantRows; ++j) {
                const int64_t t = t0 + j * step;
                v[j] = t < T ? __builtin_nontemporal_load(reinterpret_cast<const vf4*>(x + t * C + c0))
                             : vf4{0.f, 0.f, 0.f, 0.f};
            }
#pragma unroll
            for (int j = 0; j < kQuantRows; ++j) {
                const int64_t t = t0 + j * step;
                int q[4];
                const float xv[4] = {v[j].x, v[j].y, v[j].z, v[j].w};
#pragma unroll
                for (int b = 0; b < 4; ++b)
                    q[b] = s > 0.0 ? ptf_q(xv[b], s, zp, levels, al[b]) - half : zpc;
                const uint32_t pack = ((uint32_t)q[0] & 0xFFu) | (((uint32_t)q[1] & 0xFFu) << 8) |
                                      (((uint32_t)q[2] & 0xFFu) << 16) | ((uint32_t)q[3] << 24);
                if (t < T) __builtin_nontemporal_store(pack, reinterpret_cast<uint32_t*>(y + t * C + c0));
            }
        } else {
            for (int j = 0; j < kQuantRows; ++j) {
                const int64_t t = t0 + j * step;
                if (t >= T) break;
                const int64_t off = t * C + c0;
                for (int b = 0; b < 4 && c0 + b < C; ++b)
                    y[off + b] = (int8_t)(s > 0.0 ? ptf_q(x[off + b], s, zp, levels, al[b]) - half
                                                   : zpc);
            }
        }
    }
}

// y = clip(((N2 q + 2^(N1-1)) >> N1) + zp, 0, 2^b - 1) in the int8 container;
// four elements per thread when aligned.
__device__ __forceinline__ int requant_one(int32_t q, int64_t N2, int N1, int64_t zp, int64_t hi,
                                           int half) {
    const int64_t prod = N2 * (int64_t)q;
    const int64_t w = N1 > 0 ? (prod + ((int64_t)1 << (N1 - 1))) >> N1 : prod;
    const int64_t yu = w + zp;
    const int64_t yc = yu < 0 ? 0 : (yu > hi ? hi : yu);
    return (int)yc - half;
}

__global__ __launch_bounds__(kBlock) void requant_kernel(const int32_t* q, int64_t n, int64_t N2,
                                                         int N1, int zp_c, int bits, int vec4,
                                                         int8_t* y) {
    const int half = 1 << (bits - 1);
    const int64_t zp = zp_c + half;
    const int64_t hi = (1 << bits) - 1;
    const int64_t tid = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    if (vec4) {
        // four 16-byte loads in flight per thread before any is converted
        constexpr int kU = 4;
        const vi4* q4 = reinterpret_cast<const vi4*>(q);
        uint32_t* y4 = reinterpret_cast<uint32_t*>(y);
        const int64_t n4 = n / 4;
        for (int64_t i0 = tid; i0 < n4; i0 += stride * kU) {
            vi4 v[kU];
#pragma unroll
            for (int u = 0; u < kU; ++u) {
                const int64_t i = i0 + u * stride;
                v[u] = i < n4 ? __builtin_nontemporal_load(q4 + i) : vi4{0, 0, 0, 0};
            }
#pragma unroll
            for (int u = 0; u < kU; ++u) {
                const int64_t i = i0 + u * stride;
                const uint32_t p = ((uint32_t)requant_one(v[u].x, N2, N1, zp, hi, half) & 0xFFu) |
                                   (((uint32_t)requant_one(v[u].y, N2, N1, zp, hi, half) & 0xFFu) << 8) |
                                   (((uint32_t)requant_one(v[u].z, N2, N1, zp, hi, half) & 0xFFu) << 16) |
                                   ((uint32_t)requant_one(v[u].w, N2, N1, zp, hi, half) << 24);
                if (i < n4) __builtin_nontemporal_store(p, y4 + i);
            }
        }
        for (int64_t i = (n / 4) * 4 + tid; i < n; i += stride)
            y[i] = (int8_t)requant_one(q[i], N2, N1, zp, hi, half);
    } else {
        for (int64_t i = tid; i < n; i += stride)
            y[i] = (int8_t)requant_one(q[i], N2, N1, zp, hi, half);
    }
}

unsigned grid_for(int64_t work, int64_t per_block, int64_t cap) {
    const int64_t b = (work + per_block - 1) / per_block;
    return (unsigned)std::max<int64_t>(1, std::min<int64_t>(b, cap));
}

}  // namespace

template <int K>
void launch_alpha_partial(const PtfCalibArgs& a, dim3 grid, int64_t nb, double* part,
                          hipStream_t stream) {
    launch_kernel(alpha_partial_kernel<K>, grid, dim3(kBlock), 0, stream, a.x, a.T, a.C, a.bits,
                  (const double*)a.s, (const int32_t*)a.zp, nb, part);
}

hipError_t launch_ptf_calibrate(const PtfCalibArgs& a, hipStream_t stream) {
    const int64_t n = a.T * (int64_t)a.C;
    float* mm = reinterpret_cast<float*>(a.workspace);
    double* part = reinterpret_cast<double*>(mm + 2 * kMinmaxParts);
    const int vec4 = ((reinterpret_cast<uintptr_t>(a.x) & 15) == 0) ? 1 : 0;
    const unsigned nb1 = grid_for(n, (int64_t)kBlock * 16, kMinmaxParts);
    const LaunchEvents ev = launch_events();
    // the caller's events bracket the whole sequence: start on the first
    // kernel, stop on the last
    set_launch_events(ev.start, nullptr);
    launch_kernel(minmax_partial_kernel, dim3(nb1), dim3(kBlock), 0, stream, a.x, n, vec4, mm);
    set_launch_events(nullptr, nullptr);
    launch_kernel(calib_params_kernel, dim3(1), dim3(kBlock), 0, stream, (const float*)mm,
                  (int)nb1, a.bits, a.K, a.s, a.zp);
    const int64_t nb = (a.T + kPtfErrBlock - 1) / kPtfErrBlock;
    const dim3 g3((unsigned)((a.C + 63) / 64), (unsigned)nb);
    switch (a.K) {
        case 0: launch_alpha_partial<0>(a, g3, nb, part, stream); break;
        case 1: launch_alpha_partial<1>(a, g3, nb, part, stream); break;
        case 2: launch_alpha_partial<2>(a, g3, nb, part, stream); break;
        case 3: launch_alpha_partial<3>(a, g3, nb, part, stream); break;
        case 4: launch_alpha_partial<4>(a, g3, nb, part, stream); break;
        case 5: launch_alpha_partial<5>(a, g3, nb, part, stream); break;
        case 6: launch_alpha_partial<6>(a, g3, nb, part, stream); break;
        default: launch_alpha_partial<7>(a, g3, nb, part, stream); break;
    }
    const int cb = kSelChains / (a.K + 1);
    set_launch_events(nullptr, ev.stop);
    launch_kernel(alpha_select_kernel, dim3((unsigned)((a.C + cb - 1) / cb)), dim3(kBlock), 0, stream,
                  (const double*)part, a.C, a.K, nb, (const double*)a.s, a.alpha);
    set_launch_events(nullptr, nullptr);
    return hipGetLastError();
}

hipError_t launch_ptf_quantize(const PtfQuantArgs& a, hipStream_t stream) {
    const int vec4 = (a.C % 4 == 0 && (reinterpret_cast<uintptr_t>(a.x) & 15) == 0 &&
                      (reinterpret_cast<uintptr_t>(a.y) & 3) == 0)
                         ? 1
                         : 0;
    const unsigned gx = (unsigned)(((a.C + 3) / 4 + 63) / 64);
    const int64_t gy =
        std::min<int64_t>((a.T + 4 * kQuantRows - 1) / (4 * kQuantRows), std::max<int64_t>(1, 4096 / gx));
    launch_kernel(quantize_kernel, dim3(gx, (unsigned)gy), dim3(kBlock), 0, stream, a.x, a.T, a.C,
                  a.s, a.zp, a.alpha, a.bits, vec4, a.y);
    return hipGetLastError();
}

hipError_t launch_requant(const RequantArgs& a, hipStream_t stream) {
    const int vec4 = ((reinterpret_cast<uintptr_t>(a.q) & 15) == 0 &&
                      (reinterpret_cast<uintptr_t>(a.y) & 3) == 0)
                         ? 1
                         : 0;
    launch_kernel(requant_kernel, dim3(grid_for(a.n, kBlock * 16, 8192)), dim3(kBlock), 0, stream,
                  a.q, a.n, a.N2, a.N1, a.zp, a.bits, vec4, a.y);
    return hipGetLastError();
}

// Workspace of ptf_calibrate_noalloc: a fixed array on every device the
// library runs on.  In host code `scratch` names a host-side stand-in, not a
// device address: its device address is looked up per device once
// (hipGetSymbolAddress, with that device current) and only that address is
// passed to kernels.
static __device__ __align__(256) uint8_t scratch[FQ_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's address of `scratch`.
hipError_t current_scratch(void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}

}  // namespace

hipError_t launch_ptf_calibrate_noalloc(const PtfCalibArgs& a, hipStream_t stream) {
    void* ws = nullptr;
    const hipError_t e = current_scratch(&ws);
    if (e != hipSuccess) return e;
    PtfCalibArgs b = a;
    b.workspace = ws;
    return launch_ptf_calibrate(b, stream);
}

}  // namespace fqvit
