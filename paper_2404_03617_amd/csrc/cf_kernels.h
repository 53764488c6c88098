// cf_kernels.h -- host-side launcher interface between the C ABI layer
// (cf_api.hip) and the HIP kernels.  Internal; argument checking has already
// happened when these are called.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <mutex>
#include <set>
#include <utility>

namespace cf {

// Raise a kernel's dynamic-LDS limit to the 160 KB of a CU, once per (device,
// kernel) in the process; later launches of that kernel make no runtime call
// for it (the attribute is a limit, the launch still passes its own size).
inline hipError_t allow_full_lds(const void *kernel) {
    static std::mutex mu;
    static std::set<std::pair<int, const void *>> done;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return e;
    std::lock_guard<std::mutex> lk(mu);
    if (done.count({dev, kernel}))
        return hipSuccess;
    e = hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (e == hipSuccess)
        done.insert({dev, kernel});
    return e;
}

struct BlockW {
    const void *dw_w;
    const float *s0, *b0;
    const void *w1;
    const float *s1, *b1;
    const void *w2;
    const float *s2, *b2;
};

struct Shape {
    int N, H, W, C, E, k;
    int bf16;  // 0: fp16, 1: bf16
    int act;   // 0 GELU(erf), 1 ReLU, 2 identity
    int cfg = 0;  // kernel configuration (CFG_*), chosen by the autotuner
};

// Kernel configurations of the fused block (the autotuner's candidates).
enum {
    CFG_DEFAULT = 0,     // the shape's specialised kernel, full-size tiles
    CFG_GENERIC = 1,     // the generic fused kernel (cf_fused_impl.h)
    CFG_HALF_TILE = 2,   // C = 64 fp16 kernel with tiles of at most half the blocks
    CFG_TILE = 3,        // N*H*W <= 64: the tile kernels where the default is the slice kernel
    CFG_COUNT = 4
};
// Whether configuration cfg applies to shape s.
bool cfg_applies(const Shape &s, int cfg);
// Whether a tile kernel (every configuration but the slice kernel) fits the LDS for s.
bool tile_fits(const Shape &s);

// Fused block.  groups > 1 selects the hidden-split variant: partial (fp32,
// [groups][N*H*W][C]) receives each group's projection and a reduction kernel
// writes y.  Returns hipSuccess or the launch error.
hipError_t launch_fused_block(const void *x, void *y, const BlockW &w, const Shape &s,
                              int groups, float *partial, hipStream_t st);

// Small-batch hidden-split path (at most 8 tiles of 128 pixels): writes the
// groups' partials only (the caller runs the reduction), or, with one group
// and y non-null, the block output y itself.  Returns
// hipErrorInvalidConfiguration when the shape does not suit it.
hipError_t launch_small_split(const void *x, const BlockW &w, const Shape &s, int groups, float *partial,
                              hipStream_t st, void *y = nullptr);

// Block for N*H*W <= 64 (C = 128, 256, 512) without a workspace: one
// workgroup per 32 output channels, each recomputing the expand and summing
// its waves' projections in LDS.  slice_applies tells whether the shape suits
// it; launch_slice returns hipErrorInvalidConfiguration otherwise.
// the stride-2 ConvFirst block (cf_cfs2.hip)
bool convfirst_s2_supported(int H, int W, int C, int R, int K);
hipError_t launch_convfirst_s2(const void *x, void *y, const BlockW &w, int N, int H, int W, int C, int R, int K,
                               int bf16, int act, hipStream_t st);
bool slice_applies(const Shape &s);
hipError_t launch_slice(const void *x, void *y, const BlockW &w, const Shape &s, hipStream_t st);

// LDS bytes of the small-batch kernel for this shape; 0 when it does not apply.
// direct: one hidden group writing y (no tile-count limit); otherwise the
// partials of the split variant (at most 8 tiles).
size_t small_split_lds_bytes(const Shape &s, bool direct = false);

// Layer-by-layer path: depth-wise -> d, expand + act -> h, project + residual -> y.
// The depth-wise conv of a block with s0, b0: D [N][H][W][C] (cf_unfused.hip).
hipError_t launch_depthwise(const void *x, void *d, const BlockW &w, const Shape &s, hipStream_t st);

// A block as depth-wise conv, two library GEMMs and two elementwise passes
// (cf_libgemm.hip), for fp16 blocks at C = 512 over at least 4096 pixels;
// scratch holds libgemm_scratch_bytes(s) bytes, 256-byte aligned.
bool libgemm_applies(const Shape &s);
// creates the GEMM plans (outside a stream capture); false when they are missing
bool libgemm_ready(const Shape &s, hipStream_t st);
size_t libgemm_scratch_bytes(const Shape &s);
hipError_t launch_block_libgemm(const void *x, void *y, const BlockW &w, const Shape &s, void *scratch,
                                hipStream_t st);

hipError_t launch_unfused_block(const void *x, void *y, void *d, void *h, const BlockW &w,
                                const Shape &s, hipStream_t st);

// 2x2 stride-2 conv as a GEMM over the space-to-depth view of x.
hipError_t launch_downsample(const void *x, void *y, const void *wd, const float *sd,
                             const float *bd, int N, int H, int W, int Cin, int Cout, int bf16,
                             hipStream_t st);

// The paper's block: 3 x 3 grouped conv (group width 8) first, then the FFN
// and the residual.  gw [3][3][C][8]; the rest as BlockW.
struct GBlockW {
    const void *gw;
    const float *s0, *b0;
    const void *w1;
    const float *s1, *b1;
    const void *w2;
    const float *s2, *b2;
};
// The network stem in front of a grouped block: 3 x 3 stride-2 conv of the
// image x [N][Hin][Win][3] with taps w [C][3][3][3], scale/bias, ReLU.
struct StemW {
    const void *x;
    const void *w;
    const float *s, *b;
    int Hin, Win;
};
// Channel counts with a kernel: multiples of 16 from 16 to 112.
bool gblock_supported_c(int C);
// Stem + grouped block in one kernel (C = 16 or 32); s describes the block
// (H, W of the stem output).  hipErrorInvalidValue for another C.
hipError_t launch_stem_gblock(const StemW &stem, void *y, const GBlockW &w, const Shape &s, hipStream_t st);
// The stem alone: y [N][ceil(Hin/2)][ceil(Win/2)][C] (C = 16 or 32).
hipError_t launch_stem(const StemW &stem, void *y, int N, int C, int bf16, hipStream_t st);
// Fused grouped block; hipErrorInvalidValue for an unsupported C.
hipError_t launch_gblock(const void *x, void *y, const GBlockW &w, const Shape &s, hipStream_t st);

// The paper's MBConv block with Squeeze & Excitation (Sec. 5.4): expand w1
// [EC][C], grouped conv gw [3][3][EC][8], squeeze wr [R][EC], excitation we
// [EC][R], project w2 [C][EC]; fp32 scale/bias vectors, NULL meaning 1 / 0.
struct MBConvW {
    const void *w1;
    const float *s1, *b1;
    const void *gw;
    const float *s2, *b2;
    const void *wr;
    const float *br;
    const void *we;
    const float *be;
    const void *w2;
    const float *s3, *b3;
};
// K = 0: the stride-1 block (C output channels, residual); K > 0: the
// stride-2 block (BlurPool after the grouped conv, K output channels on a
// ceil(H/2) x ceil(W/2) map, no residual).
// Shapes with a kernel: H, W <= 16 (>= 2 for stride 2), C % 16 == 0,
// E*C % 64 == 0, E*C <= 4096, 1 <= R <= 256, K % 16 == 0.
bool mbconv_supported(int H, int W, int C, int E, int R, int K = 0);
// Images the device can hold in flight at once (all their work items resident).
hipError_t mbconv_resident_slots(int H, int W, int C, int E, int R, int K, int bf16, int *slots);
// Workspace bytes for `slots` images in flight.
size_t mbconv_workspace_bytes(int N, int H, int W, int C, int E, int R, int K, int slots);
// Fused MBConv block; ws of ws_bytes >= mbconv_workspace_bytes(..., 1)
// (hipErrorInvalidValue otherwise), its header zero.  The first int of ws is
// set if a barrier wait gave up.  coop: hipLaunchCooperativeKernel, else an
// ordinary launch of the same grid.
hipError_t launch_mbconv(const void *x, void *y, const MBConvW &w, int N, int H, int W, int C, int E, int R, int K,
                         int bf16, void *ws, size_t ws_bytes, bool coop, hipStream_t st);

// Upper bound of dynamic LDS the fused kernel needs for this shape (bytes);
// 0 when no kernel configuration fits.
size_t fused_lds_bytes(const Shape &s);

// Number of compute units of the current device (cached per device).
int device_cu_count();

}  // namespace cf
