// cf_gblock_c112.hip -- the grouped-conv ConvFirst block for C = 112 (one unit per
// channel count so the instantiations compile in parallel).
#include "cf_gblock.h"

namespace cf {
hipError_t launch_gblock_c112(const void *x, void *y, const GBlockW &w, const Shape &s, hipStream_t st) {
    return gblk::launch_c<112>(x, y, w, s, st);
}
}  // namespace cf
