// Test-only stand-ins for the kernel launchers of libfqvit.  The C ABI's host
// code (argument validation, the I-Exp integer constants, the dyadic
// multiplier of the requantization) is linked against these in the CPU
// sanitizer build (tests/test_sanitizers.py), so every entry point can run to
// its launch without a GPU.  Each stub counts its call and launches nothing.
#include "fqvit_internal.h"

namespace fqvit {

static int g_launches = 0;

hipError_t launch_ptf_layernorm(const LnArgs&, hipStream_t) { ++g_launches; return hipSuccess; }
hipError_t launch_lis(const LisArgs&, hipStream_t) { ++g_launches; return hipSuccess; }
hipError_t launch_lis_qk(const LisArgs&, const QkInput&, hipStream_t) {
    ++g_launches;
    return hipSuccess;
}
hipError_t launch_attn_v_shift(const AvArgs&, hipStream_t) { ++g_launches; return hipSuccess; }
hipError_t launch_attn_v_shift_wide(const AvWideArgs&, hipStream_t) { ++g_launches; return hipSuccess; }
hipError_t launch_ptf_calibrate(const PtfCalibArgs&, hipStream_t) { ++g_launches; return hipSuccess; }
hipError_t launch_ptf_calibrate_noalloc(const PtfCalibArgs& a, hipStream_t) {
    ++g_launches;
    return a.workspace == nullptr ? hipSuccess : hipErrorInvalidValue;
}
hipError_t launch_ptf_quantize(const PtfQuantArgs&, hipStream_t) { ++g_launches; return hipSuccess; }
hipError_t launch_requant(const RequantArgs&, hipStream_t) { ++g_launches; return hipSuccess; }

}  // namespace fqvit

extern "C" int fq_test_launch_count(void) { return fqvit::g_launches; }
