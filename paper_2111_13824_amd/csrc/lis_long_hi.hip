// Instantiations of the long-row Log-Int-Softmax attention kernel for 15..20
// chunks of 32 keys.
#include "lis_long.h"

namespace fqvit {
namespace lis {

hipError_t launch_lis_long_hi(int nc, int dtm, bool half, const LisArgs& a, const LisLaunch& p,
                              size_t lds, hipStream_t stream) {
    switch (nc) {
        case 15: return launch_long_nc<15>(dtm, half, a, p, lds, stream);
        case 16: return launch_long_nc<16>(dtm, half, a, p, lds, stream);
        case 17: return launch_long_nc<17>(dtm, half, a, p, lds, stream);
        case 18: return launch_long_nc<18>(dtm, half, a, p, lds, stream);
        case 19: return launch_long_nc<19>(dtm, half, a, p, lds, stream);
        case 20: return launch_long_nc<20>(dtm, half, a, p, lds, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace lis
}  // namespace fqvit
