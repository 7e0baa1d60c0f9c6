// Instantiations of the register-resident Log-Int-Softmax kernels for 11..20
// chunks of 32 keys.
#include "lis_device.h"

namespace fqvit {
namespace lis {

hipError_t launch_lis_regs_hi(int nc, bool fused, bool multi, int dtm, bool pre0,
                              const LisArgs& a, const LisLaunch& p, dim3 grid, size_t lds,
                              hipStream_t stream) {
    switch (nc) {
        case 11: return launch_lis_nc<11>(fused, multi, dtm, pre0, a, p, grid, lds, stream);
        case 12: return launch_lis_nc<12>(fused, multi, dtm, pre0, a, p, grid, lds, stream);
        case 13: return launch_lis_nc<13>(fused, multi, dtm, pre0, a, p, grid, lds, stream);
        case 14: return launch_lis_nc<14>(fused, multi, dtm, pre0, a, p, grid, lds, stream);
        case 15: return launch_lis_nc<15>(fused, multi, dtm, pre0, a, p, grid, lds, stream);
        case 16: return launch_lis_nc<16>(fused, multi, dtm, pre0, a, p, grid, lds, stream);
        case 17: return launch_lis_nc<17>(fused, multi, dtm, pre0, a, p, grid, lds, stream);
        case 18: return launch_lis_nc<18>(fused, multi, dtm, pre0, a, p, grid, lds, stream);
        case 19: return launch_lis_nc<19>(fused, multi, dtm, pre0, a, p, grid, lds, stream);
        case 20: return launch_lis_nc<20>(fused, multi, dtm, pre0, a, p, grid, lds, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace lis
}  // namespace fqvit
