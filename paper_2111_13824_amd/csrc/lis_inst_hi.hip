// Instantiations of the Log-Int-Softmax tile kernels for 11..20 chunks of
// 32 keys.
#include "lis_device.h"

namespace fqvit {
namespace lis {

hipError_t launch_lis_regs_hi(int nc, bool fused, int dtm, bool fp, const LisArgs& a,
                              const LisLaunch& p, dim3 grid, size_t lds, hipStream_t stream) {
    switch (nc) {
        case 11: return launch_lis_nc<11>(fused, dtm, fp, a, p, grid, lds, stream);
        case 12: return launch_lis_nc<12>(fused, dtm, fp, a, p, grid, lds, stream);
        case 13: return launch_lis_nc<13>(fused, dtm, fp, a, p, grid, lds, stream);
        case 14: return launch_lis_nc<14>(fused, dtm, fp, a, p, grid, lds, stream);
        case 15: return launch_lis_nc<15>(fused, dtm, fp, a, p, grid, lds, stream);
        case 16: return launch_lis_nc<16>(fused, dtm, fp, a, p, grid, lds, stream);
        case 17: return launch_lis_nc<17>(fused, dtm, fp, a, p, grid, lds, stream);
        case 18: return launch_lis_nc<18>(fused, dtm, fp, a, p, grid, lds, stream);
        case 19: return launch_lis_nc<19>(fused, dtm, fp, a, p, grid, lds, stream);
        case 20: return launch_lis_nc<20>(fused, dtm, fp, a, p, grid, lds, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace lis
}  // namespace fqvit
