// Instantiations of the Log-Int-Softmax tile kernels for 1..10 chunks of
// 32 keys.
#include "lis_device.h"

namespace fqvit {
namespace lis {

hipError_t launch_lis_regs_lo(int nc, bool fused, int dtm, bool fp, const LisArgs& a,
                              const LisLaunch& p, dim3 grid, size_t lds, hipStream_t stream) {
    switch (nc) {
        case 1: return launch_lis_nc<1>(fused, dtm, fp, a, p, grid, lds, stream);
        case 2: return launch_lis_nc<2>(fused, dtm, fp, a, p, grid, lds, stream);
        case 3: return launch_lis_nc<3>(fused, dtm, fp, a, p, grid, lds, stream);
        case 4: return launch_lis_nc<4>(fused, dtm, fp, a, p, grid, lds, stream);
        case 5: return launch_lis_nc<5>(fused, dtm, fp, a, p, grid, lds, stream);
        case 6: return launch_lis_nc<6>(fused, dtm, fp, a, p, grid, lds, stream);
        case 7: return launch_lis_nc<7>(fused, dtm, fp, a, p, grid, lds, stream);
        case 8: return launch_lis_nc<8>(fused, dtm, fp, a, p, grid, lds, stream);
        case 9: return launch_lis_nc<9>(fused, dtm, fp, a, p, grid, lds, stream);
        case 10: return launch_lis_nc<10>(fused, dtm, fp, a, p, grid, lds, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace lis
}  // namespace fqvit
