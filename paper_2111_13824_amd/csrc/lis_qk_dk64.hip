// Instantiations of the integer-only attention kernel for a 64-byte feature
// dimension of Q and K.
#include "lis_qk_kernel.h"

namespace fqvit {
namespace lis {

hipError_t launch_qk_dk64(int nc, int dtm, bool half, int fp, const LisArgs& a, const QkArgs& qa,
                          const LisLaunch& p, size_t lds, hipStream_t stream) {
    return launch_qk_dk<64>(nc, dtm, half, fp, a, qa, p, lds, stream);
}

}  // namespace lis
}  // namespace fqvit
