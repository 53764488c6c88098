// cf_gblock.hip -- dispatch of the grouped-conv ConvFirst block (the paper's
// own block, Sec. 5.3) to its per-channel-count instantiations.
#include "cf_kernels.h"

namespace cf {

hipError_t launch_gblock_c16(const void *, void *, const GBlockW &, const Shape &, hipStream_t);
hipError_t launch_gblock_c32(const void *, void *, const GBlockW &, const Shape &, hipStream_t);
hipError_t launch_gblock_c48(const void *, void *, const GBlockW &, const Shape &, hipStream_t);
hipError_t launch_gblock_c64(const void *, void *, const GBlockW &, const Shape &, hipStream_t);
hipError_t launch_gblock_c80(const void *, void *, const GBlockW &, const Shape &, hipStream_t);
hipError_t launch_gblock_c96(const void *, void *, const GBlockW &, const Shape &, hipStream_t);
hipError_t launch_gblock_c112(const void *, void *, const GBlockW &, const Shape &, hipStream_t);

bool gblock_supported_c(int C) { return C >= 16 && C <= 112 && C % 16 == 0; }

hipError_t launch_gblock(const void *x, void *y, const GBlockW &w, const Shape &s, hipStream_t st) {
    switch (s.C) {
    case 16: return launch_gblock_c16(x, y, w, s, st);
    case 32: return launch_gblock_c32(x, y, w, s, st);
    case 48: return launch_gblock_c48(x, y, w, s, st);
    case 64: return launch_gblock_c64(x, y, w, s, st);
    case 80: return launch_gblock_c80(x, y, w, s, st);
    case 96: return launch_gblock_c96(x, y, w, s, st);
    case 112: return launch_gblock_c112(x, y, w, s, st);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace cf
