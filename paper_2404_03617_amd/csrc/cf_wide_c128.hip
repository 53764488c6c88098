// cf_wide_c128.hip -- fused block kernel for C = 128 (see cf_wide.h).
#include "cf_wide.h"

namespace cf {
hipError_t launch_wide_c128(const void *x, void *y, const BlockW &w, const Shape &s, hipStream_t st) {
    return wide::launch_c<128>(x, y, w, s, st);
}
}  // namespace cf
