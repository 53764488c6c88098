// cf_wide_c512.hip -- fused block kernel for C = 512 (see cf_wide.h).
#include "cf_wide.h"

namespace cf {
hipError_t launch_wide_c512(const void *x, void *y, const BlockW &w, const Shape &s, int groups, float *partial,
                            hipStream_t st) {
    return wide::launch_c512(x, y, w, s, groups, partial, st);
}
}  // namespace cf
