// Fused-block kernel instantiations for C = 256, F16 I/O.
#include "cf_fused_impl.h"

namespace cf {
namespace fused {
hipError_t launch_c256_F16(const FusedArgs &a, int k, int act, int groups, hipStream_t st) {
    return launch_ct<256, F16>(a, k, act, groups, st);
}
}  // namespace fused
}  // namespace cf
