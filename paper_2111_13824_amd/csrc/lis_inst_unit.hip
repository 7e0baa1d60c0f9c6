// Instantiations of the Log-Int-Softmax unit kernels for 1..7 chunks of 32 keys.
#include "lis_device.h"

namespace fqvit {
namespace lis {

static_assert(kUnitMaxNC == 7, "instantiated chunk counts");

hipError_t launch_lis_unit(int nc, bool fused, int dtm, bool half, int wpu, const LisArgs& a,
                           const LisLaunch& p, size_t lds, hipStream_t stream) {
    switch (nc) {
        case 1: return launch_unit_nc<1>(fused, dtm, half, wpu, a, p, lds, stream);
        case 2: return launch_unit_nc<2>(fused, dtm, half, wpu, a, p, lds, stream);
        case 3: return launch_unit_nc<3>(fused, dtm, half, wpu, a, p, lds, stream);
        case 4: return launch_unit_nc<4>(fused, dtm, half, wpu, a, p, lds, stream);
        case 5: return launch_unit_nc<5>(fused, dtm, half, wpu, a, p, lds, stream);
        case 6: return launch_unit_nc<6>(fused, dtm, half, wpu, a, p, lds, stream);
        case 7: return launch_unit_nc<7>(fused, dtm, half, wpu, a, p, lds, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace lis
}  // namespace fqvit
