// Fused Log-Int-Softmax + BitShift Attn x V for long rows (Supplement A.2,
// Alg. 1 and 2; Sec. 3.3 and its Fig. 4) on gfx950: rows of 10 to 20 chunks of
// 32 keys (289 to 640 keys), d <= 64, float path.
//
// One workgroup of kLongWaves wavefronts per attention unit.  The unit's V^T
// is staged once in LDS (bf16, keys in the MFMA order of lis_device.h), and so
// is a table of the I-Exp value e(u) (its binary32 bits) for every clamped
// input u in [0, n |q_ln2|]: one lookup replaces the integer steps of
// iexp_fu.  Each wavefront walks the unit's 16-row tiles and reads every
// logit once:
//   * load: lane (r, kg) keeps its 8 keys of every chunk as 16-bit values
//     d = v - m0, m0 the row's maximum over its first chunk (saturated to
//     16 bits; the row maximum is m0 + delta with delta = max d).  When
//     delta <= 32767 no kept value saturated upwards, and a value saturated
//     downwards lies more than 32767 >= n |q_ln2| below the maximum, where
//     I-Exp clamps anyway, so u = min(delta - d, n |q_ln2|) is exact.  A tile
//     with a larger delta in any of its rows is computed from the logits
//     again (long_tile_exact);
//   * u is stored back as the byte offset 4 u of its table entry;
//   * sum: e = table[u], the row sum S in binary64 (exact: integers below
//     2^52);
//   * codes: the table entry again, the code by code_rev_f, P = 2^(N - code)
//     as bf16 bits, and the chunk's MFMA with V^T (exact, see lis_device.h).
// The next tile's logits are loaded during the code pass of the current one,
// one chunk per chunk computed, into the registers that chunk frees.  Logits
// and bias are read as buffer loads over the unit's planes: a load that is
// not needed (no next tile) addresses past the buffer and returns 0 without a
// memory access, so every load is issued unconditionally.
#pragma once

#include "lis_device.h"

namespace fqvit {
namespace lis {

// Measured on ViT-L/16 at 384 px (256 x 577 x 577, one MI355X): 8 wavefronts
// with 2, 4, 6 or 8 chunks in flight 122-131 us, all within noise of each
// other; 12 wavefronts (168 VGPRs) spill 115 to 172 registers.
constexpr int kLongWaves = 8;                  // 2 wavefronts per SIMD (256 VGPRs)
constexpr int kLongPF = 4;                     // chunks in flight per wavefront
constexpr int kLongMinNC = 10;
constexpr int kLongMaxNC = 20;

typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

struct LongRows {
    __amdgpu_buffer_rsrc_t lg;     // the unit's logits [Lq, Lk]
    __amdgpu_buffer_rsrc_t bs;     // its head's bias plane [Lq, Lk] (unused without bias)
    bool bias;
};

// The 8 logits (+ bias) of lane (r, kg) in chunk c of the row at byte offset
// roff of the unit's planes; roff < 0: nothing needed (every load past the
// buffers, no memory access).  Keys past Lk hold arbitrary values.
__device__ __forceinline__ void long_load(int (&dst)[8], const LongRows& lr, int roff, int c,
                                          int kg) {
    const int o0 = roff < 0 ? INT_MIN : roff + 4 * (32 * c + 4 * kg);
    const int o1 = roff < 0 ? INT_MIN : o0 + 64;
    const i32x4a4 x = __builtin_bit_cast(i32x4a4, __builtin_amdgcn_raw_buffer_load_b128(lr.lg, o0, 0, 0));
    const i32x4a4 y = __builtin_bit_cast(i32x4a4, __builtin_amdgcn_raw_buffer_load_b128(lr.lg, o1, 0, 0));
    dst[0] = x.x; dst[1] = x.y; dst[2] = x.z; dst[3] = x.w;
    dst[4] = y.x; dst[5] = y.y; dst[6] = y.z; dst[7] = y.w;
    if (lr.bias) {
        const i32x4a4 bx = __builtin_bit_cast(i32x4a4, __builtin_amdgcn_raw_buffer_load_b128(lr.bs, o0, 0, 0));
        const i32x4a4 by = __builtin_bit_cast(i32x4a4, __builtin_amdgcn_raw_buffer_load_b128(lr.bs, o1, 0, 0));
        dst[0] += bx.x; dst[1] += bx.y; dst[2] += bx.z; dst[3] += bx.w;
        dst[4] += by.x; dst[5] += by.y; dst[6] += by.z; dst[7] += by.w;
    }
}

// Chunk c's keys as 16-bit d = v - m0 (saturated) into pk[4], the pairs
// (0,1) .. (6,7); masked keys (last chunk, bit t of valid clear) as -32768 and
// out of the maximum.  rmax: the lane's largest d so far.
template <bool LAST>
__device__ __forceinline__ void long_convert(uint32_t (&pk)[4], const int (&x)[8], int m0, int& rmax,
                                             uint32_t valid) {
    int d[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) {
        d[t] = x[t] - m0;
        if (LAST) d[t] = ((valid >> t) & 1u) ? d[t] : -32768;
    }
#pragma unroll
    for (int t = 0; t < 8; t += 2) rmax = max(rmax, max(d[t], d[t + 1]));
#pragma unroll
    for (int w = 0; w < 4; ++w)
        pk[w] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pk_i16(d[2 * w], d[2 * w + 1]));
}

// Loads and converts all NC chunks of one tile (a window of PF chunks in
// flight); returns the row's delta (lane-group uniform).
template <int NC, int PF>
__device__ __forceinline__ int long_load_tile(uint32_t (&pk)[NC][4], const LongRows& lr, int roff,
                                              int kg, uint32_t valid) {
    int raw[PF][8];
#pragma unroll
    for (int q = 0; q < PF; ++q) long_load(raw[q], lr, roff, q, kg);
    int m0 = 0, rmax = INT_MIN;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        if (c == 0) {
            int mx = raw[0][0];
#pragma unroll
            for (int t = 1; t < 8; ++t) mx = max(mx, raw[0][t]);
            m0 = row4_max(mx);
        }
        if (c == NC - 1) long_convert<true>(pk[c], raw[c % PF], m0, rmax, valid);
        else long_convert<false>(pk[c], raw[c % PF], m0, rmax, valid);
        if (c + PF < NC) long_load(raw[c % PF], lr, roff, c + PF, kg);
    }
    return row4_max(rmax);
}

// V^T of a whole unit (keys [0, kp), kp a multiple of 32) staged by a workgroup
// of NTHREADS threads, as stage_store does: item = (16-column group, key quad).
template <int DTMAX, int NTHREADS>
__device__ __forceinline__ void long_stage_vt(uint16_t* vt, int ld, const int8_t* vg, int Lk, int d,
                                              int kp, int zp, bool vec_ok) {
    const int nquads = kp / 4;
    const float off = (float)(128 + zp);
    for (int idx = threadIdx.x; idx < nquads * DTMAX; idx += NTHREADS) {
        const int cg = idx / nquads;
        const int jj = 4 * (idx - cg * nquads);
        const int dd = 16 * cg;
        u32x4 w[4];
#pragma unroll
        for (int t = 0; t < 4; ++t)
            w[t] = (dd < d && jj + t < Lk) ? load_v16(vg + (int64_t)(jj + t) * d, dd, d, vec_ok)
                                           : u32x4{0u, 0u, 0u, 0u};
        const int pos = (jj & ~31) + chunk_pos(jj & 31);
#pragma unroll
        for (int t = 0; t < 4; ++t) w[t] ^= 0x80808080u;
#pragma unroll
        for (int q = 0; q < 16; ++q) {
            float f[4];
#pragma unroll
            for (int t = 0; t < 4; ++t) f[t] = (float)((w[t][q >> 2] >> (8 * (q & 3))) & 0xFFu) - off;
            *reinterpret_cast<u32x2*>(vt + (16 * cg + q) * ld + pos) =
                u32x2{bf16_pair(f[0], f[1]), bf16_pair(f[2], f[3])};
        }
    }
}

// e (binary32 bits) of the table entry at byte offset off
__device__ __forceinline__ uint32_t long_table(const uint8_t* smem, uint32_t off) {
    return *reinterpret_cast<const uint32_t*>(smem + off);
}

// A tile whose rows span more than 32767 logit units: max, sum and code
// passes over the logits in memory (the rows of lane group r at row pointers
// rp), the same arithmetic as the stream kernel's float path.
template <int NC, int DTMAX, bool HALF>
__device__ void long_tile_exact(f32x4 (&acc)[DTMAX], const RowPtrs& rp, const LisConsts& k,
                                const uint16_t* vt, int ld, int Lk, int r, int kg) {
    int mx = INT_MIN;
#pragma unroll 1
    for (int c = 0; c < NC; ++c) {
        int lg[8];
        load_chunk<false>(lg, rp.row, rp.brow, c, kg, Lk, rp.tail_vec);
#pragma unroll
        for (int t = 0; t < 8; ++t) mx = max(mx, lg[t]);
    }
    mx = row4_max(mx);
    double part[2] = {0.0, 0.0};
#pragma unroll 1
    for (int c = 0; c < NC; ++c) {
        int lg[8];
        load_chunk<false>(lg, rp.row, rp.brow, c, kg, Lk, rp.tail_vec);
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            const float e = iexp_f(lg[t], mx, k);
            part[t & 1] += lg[t] != INT_MIN ? (double)e : 0.0;
        }
    }
    RowState st;
    const double S2 = 2.0 * row4_sum(part[0] + part[1]);
    st.S2s = S2 * kCodeScale;
    st.sc = kCodeScale;
    asm volatile("" : "+s"(st.sc));
    st.tau = third_floor_f32(S2);
    const uint32_t kr = ((uint32_t)(k.top + 1) << 25) - 1u;
#pragma unroll 1
    for (int c = 0; c < NC; ++c) {
        int lg[8];
        load_chunk<false>(lg, rp.row, rp.brow, c, kg, Lk, rp.tail_vec);
        uint32_t ex[8];
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            const bool valid = lg[t] != INT_MIN;
            const int eb = __float_as_int(iexp_f(valid ? lg[t] : mx, mx, k));
            ex[t] = valid ? 127u + code_rev_f(eb, st, kr) : 0u;
        }
        const u32x4 pb = {(ex[0] | (ex[1] << 16)) << 7, (ex[2] | (ex[3] << 16)) << 7,
                          (ex[4] | (ex[5] << 16)) << 7, (ex[6] | (ex[7] << 16)) << 7};
        if (HALF && c == NC - 1) chunk_mfma<DTMAX, true>(acc, pb, vt, ld, c, r, kg);
        else chunk_mfma<DTMAX, false>(acc, pb, vt, ld, c, r, kg);
    }
}

// WAVES wavefronts per workgroup, PF chunks in flight per wavefront.
template <int NC, int DTMAX, bool HALF, int WAVES, int PF>
__global__ __launch_bounds__(64 * WAVES) void lis_long_kernel(LisArgs a, LisLaunch p) {
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    // LDS: the I-Exp table at offset 0 (so that 4 u is its entry's address),
    // then V^T
    uint32_t* tab = reinterpret_cast<uint32_t*>(smem);
    uint16_t* vt = reinterpret_cast<uint16_t*>(smem + p.tab_bytes);
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

    long_stage_vt<DTMAX, 64 * WAVES>(vt, p.ld, a.v + g * (int64_t)Lk * a.d, Lk, a.d, 32 * NC, a.zp_v,
                                     p.vec_ok);
    for (uint32_t u = threadIdx.x; u <= k.u_max; u += 64 * WAVES) tab[u] = __float_as_uint(iexp_fu(u, k));
    __syncthreads();

    LongRows lr;
    const int plane = a.Lq * Lk * 4;       // bytes of one unit's plane (< 2^31)
    lr.lg = __builtin_amdgcn_make_buffer_rsrc((void*)(a.logits + g * a.Lq * (int64_t)Lk), (short)0,
                                              plane, 0x00020000);
    lr.bias = a.bias != nullptr;
    lr.bs = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(a.bias ? a.bias + (g % a.Hb) * a.Lq * (int64_t)Lk : a.logits), (short)0,
        lr.bias ? plane : 0, 0x00020000);
    UnitBase ub;
    ub.loff = g * a.Lq * (int64_t)Lk;
    ub.boff = a.bias ? (g % a.Hb) * a.Lq * (int64_t)Lk : 0;

    // keys of the last chunk that exist: bit t for key 32 (NC - 1) + 4 kg + t
    // (t < 4) or + 12 + t (t >= 4)
    uint32_t valid = 0;
#pragma unroll
    for (int t = 0; t < 8; ++t)
        valid |= (32 * (NC - 1) + 4 * kg + (t < 4 ? t : t + 12) < Lk ? 1u : 0u) << t;
    const uint32_t kr = ((uint32_t)(k.top + 1) << 25) - 1u;
    const u16x2 umax2 = {(unsigned short)k.u_max, (unsigned short)k.u_max};

    uint32_t pk[NC][4];
    int delta = 0;
    bool have = false;
    for (int tile = wave; tile < p.ntiles; tile += WAVES) {
        const int i0 = 16 * tile;
        const int i = min(i0 + r, a.Lq - 1);
        if (!have) delta = long_load_tile<NC, PF>(pk, lr, i * Lk * 4, kg, valid);
        const int next = tile + WAVES;
        const bool has_next = next < p.ntiles;
        f32x4 acc[DTMAX];
#pragma unroll
        for (int dt = 0; dt < DTMAX; ++dt) acc[dt] = f32x4{0.f, 0.f, 0.f, 0.f};

        if (__ballot(delta > 32767) != 0) {
            // some row spans more than 16 bits: from the logits again
            long_tile_exact<NC, DTMAX, HALF>(acc, unit_row<NC>(a, p, ub, i), k, vt, p.ld, Lk, r, kg);
            store_out<DTMAX>(acc, a, g, i0, r, kg);
            have = false;
            continue;
        }

        // d -> byte offset 4 min(delta - d, n |q_ln2|) of the table entry
        const u16x2 dd2 = {(unsigned short)delta, (unsigned short)delta};
#pragma unroll
        for (int c = 0; c < NC; ++c) {
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                const u16x2 x = __builtin_bit_cast(u16x2, pk[c][w]);
                const u16x2 u = __builtin_elementwise_min((u16x2)(dd2 - x), umax2);
                pk[c][w] = __builtin_bit_cast(uint32_t, (u16x2)(u << (unsigned short)2));
            }
        }

        // row sum: four exact binary64 partial sums
        double part[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
        for (int c = 0; c < NC; ++c) {
#pragma unroll
            for (int t = 0; t < 8; ++t) {
                const uint32_t off = (t & 1) ? pk[c][t >> 1] >> 16 : pk[c][t >> 1] & 0xFFFFu;
                float e = __uint_as_float(long_table(smem, off));
                if (c == NC - 1) e = ((valid >> t) & 1u) ? e : 0.0f;
                part[t & 3] += (double)e;
            }
            // one chunk's table reads at a time (hoisting them all would
            // take a register per key)
            __builtin_amdgcn_sched_barrier(0);
        }
        RowState st;
        {
            double sum = (part[0] + part[1]) + (part[2] + part[3]);
            sum = row4_sum(sum);
            const double S2 = 2.0 * sum;
            st.S2s = S2 * kCodeScale;
            st.sc = kCodeScale;
            asm volatile("" : "+s"(st.sc));
            st.tau = third_floor_f32(S2);
        }

        // codes and the product, the next tile streaming in
        const int inext = min(16 * next + r, a.Lq - 1);
        const int roffn = has_next ? inext * Lk * 4 : -1;
        int raw[PF][8];
#pragma unroll
        for (int q = 0; q < PF; ++q) long_load(raw[q], lr, roffn, q, kg);
        int m0n = 0, rmaxn = INT_MIN;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            uint32_t ex[8];
#pragma unroll
            for (int t = 0; t < 8; ++t) {
                const uint32_t off = (t & 1) ? pk[c][t >> 1] >> 16 : pk[c][t >> 1] & 0xFFFFu;
                const uint32_t x = 127u + code_rev_f((int)long_table(smem, off), st, kr);
                ex[t] = (c == NC - 1 && !((valid >> t) & 1u)) ? 0u : x;
            }
            const u32x4 pb = {(ex[0] | (ex[1] << 16)) << 7, (ex[2] | (ex[3] << 16)) << 7,
                              (ex[4] | (ex[5] << 16)) << 7, (ex[6] | (ex[7] << 16)) << 7};
            if (HALF && c == NC - 1) chunk_mfma<DTMAX, true>(acc, pb, vt, p.ld, c, r, kg);
            else chunk_mfma<DTMAX, false>(acc, pb, vt, p.ld, c, r, kg);
            // the next tile's chunk c - PF + 1 into the registers chunk
            // c has just freed
            const int j = c - PF + 1 >= 0 ? c - PF + 1 : 0;
            if (c - PF + 1 >= 0) {
                if (j == 0) {
                    int mx = raw[0][0];
#pragma unroll
                    for (int t = 1; t < 8; ++t) mx = max(mx, raw[0][t]);
                    m0n = row4_max(mx);
                }
                if (j == NC - 1) long_convert<true>(pk[j], raw[j % PF], m0n, rmaxn, valid);
                else long_convert<false>(pk[j], raw[j % PF], m0n, rmaxn, valid);
                if (j + PF < NC) long_load(raw[j % PF], lr, roffn, j + PF, kg);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (int j = NC - PF + 1; j < NC; ++j) {
            if (j == NC - 1) long_convert<true>(pk[j], raw[j % PF], m0n, rmaxn, valid);
            else long_convert<false>(pk[j], raw[j % PF], m0n, rmaxn, valid);
        }
        store_out<DTMAX>(acc, a, g, i0, r, kg);
        delta = row4_max(rmaxn);
        have = has_next;
    }
}

// Launch for exactly NC chunks (kLongMinNC <= NC <= kLongMaxNC), DTMAX 2 or 4.
template <int NC, int WAVES = kLongWaves, int PF = kLongPF>
hipError_t launch_long_nc(int dtm, bool half, const LisArgs& a, const LisLaunch& p, size_t lds,
                          hipStream_t s) {
#define FQ_LONG(DTM, HALF)                                                              \
    launch_kernel(lis_long_kernel<NC, DTM, HALF, WAVES, PF>, dim3((unsigned)a.G),         \
                  dim3(64 * WAVES), lds, s, a, p)
    if (dtm == 2) {
        if (half) FQ_LONG(2, true);
        else FQ_LONG(2, false);
    } else {
        if (half) FQ_LONG(4, true);
        else FQ_LONG(4, false);
    }
#undef FQ_LONG
    return hipGetLastError();
}

// Per chunk-count launchers, instantiated in lis_long_lo.hip (10..14) and
// lis_long_hi.hip (15..20).
hipError_t launch_lis_long_lo(int nc, int dtm, bool half, const LisArgs& a, const LisLaunch& p,
                              size_t lds, hipStream_t stream);
hipError_t launch_lis_long_hi(int nc, int dtm, bool half, const LisArgs& a, const LisLaunch& p,
                              size_t lds, hipStream_t stream);

}  // namespace lis
}  // namespace fqvit
