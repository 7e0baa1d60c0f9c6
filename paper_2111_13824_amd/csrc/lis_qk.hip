// Host side of the integer-only attention from int8 Q and K (kernels in
// lis_qk_kernel.h and lis_qk_long.hip): launch geometry and LDS of one
// workgroup per unit.
#include "lis_qk_kernel.h"

namespace fqvit {

hipError_t launch_lis_qk(const LisArgs& a, const QkInput& in, hipStream_t stream) {
    using namespace lis;
    const int nc = (a.Lk + 31) / 32;
    int dt = 2;
    while (16 * dt < a.d) dt <<= 1;
    LisLaunch p{};
    p.ntiles = (a.Lq + 15) / 16;
    p.dpad = 16 * dt;
    p.ncg = dt;
    p.kb = 32 * nc;
    p.ld = p.kb + 8;
    p.vec_ok = (a.d % 16 == 0) && ((reinterpret_cast<uintptr_t>(a.v) & 15) == 0);
    p.vt_bytes = p.dpad * p.ld * (int)sizeof(uint16_t);
    // output rows as 16-byte units (d % 4 == 0 and a 16-byte aligned out)
    p.out_vec = (a.d % 4 == 0) && ((reinterpret_cast<uintptr_t>(a.out) & 15) == 0);
    p.n_logits = 0;
    p.n_bias = a.bias ? (int64_t)a.Hb * a.Lq * a.Lk : 0;
    const size_t lds = (size_t)p.vt_bytes + (size_t)32 * nc * in.dk + (size_t)32 * nc * sizeof(int32_t);
    const bool half = a.Lk - 32 * (nc - 1) <= 16;
    // float path (and its I-Exp without the pre-shift where that is 0) or the
    // integer path
    const int fp = a.k.fp_ok != 0 ? (a.k.pre == 0 ? 2 : 1) : 0;
    const QkArgs qa{in.q, in.k, in.zp_q, in.zp_k};
    // rows beyond 7 chunks: logits recomputed per pass from K in LDS
    if (nc > 7) return launch_qk_long(in.dk, dt, fp, a, qa, p, lds, stream);
    if (in.dk == 32) return launch_qk_dk32(nc, dt, half, fp, a, qa, p, lds, stream);
    return launch_qk_dk64(nc, dt, half, fp, a, qa, p, lds, stream);
}

}  // namespace fqvit
