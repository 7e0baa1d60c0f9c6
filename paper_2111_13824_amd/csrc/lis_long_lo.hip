// Instantiations of the long-row Log-Int-Softmax attention kernel for 10..14
// chunks of 32 keys.
#include "lis_long.h"

namespace fqvit {
namespace lis {

hipError_t launch_lis_long_lo(int nc, int dtm, bool half, const LisArgs& a, const LisLaunch& p,
                              size_t lds, hipStream_t stream) {
    switch (nc) {
        case 10: return launch_long_nc<10>(dtm, half, a, p, lds, stream);
        case 11: return launch_long_nc<11>(dtm, half, a, p, lds, stream);
        case 12: return launch_long_nc<12>(dtm, half, a, p, lds, stream);
        case 13: return launch_long_nc<13>(dtm, half, a, p, lds, stream);
        case 14: return launch_long_nc<14>(dtm, half, a, p, lds, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace lis
}  // namespace fqvit
