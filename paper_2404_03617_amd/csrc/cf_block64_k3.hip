// cf_block64_k3.hip -- C = 64 fused block kernel, 3x3 depth-wise (see cf_block64.h).
#include "cf_block64.h"

namespace cf {
hipError_t launch_block64_k3(const void *x, void *y, const BlockW &w, const Shape &s, hipStream_t st) {
    return b64::launch_k<3>(x, y, w, s, st);
}
}  // namespace cf
