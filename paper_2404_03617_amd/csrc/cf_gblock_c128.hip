// cf_gblock_c128.hip -- the grouped-conv ConvFirst block for C = 128 (one unit per
// channel count so the instantiations compile in parallel).
#include "cf_gblock.h"

namespace cf {
hipError_t launch_gblock_c128(const void *x, void *y, const GBlockW &w, const Shape &s, hipStream_t st) {
    return gblk::launch_c<128>(x, y, w, s, st);
}
}  // namespace cf
