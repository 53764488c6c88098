// cf_fused.hip -- dispatch of the ConvFirst block-fusion kernels (Sec. 5.3.1,
// Sec. 5.5.1 of Lavin, arXiv:2404.03617) and the hidden-split reduction.
//
// Every fused kernel evaluates the whole residual block for a range of
// 32-pixel blocks of the flattened N*H*W index: halo rows into LDS, k x k
// depth-wise conv on the VALU, then a loop over chunks of 32 hidden channels
// (eq. e:ffn-eff) with expand and project on v_mfma_f32_32x32x16, phi in
// between, and one store of the output tile.  The hidden values never reach
// device memory.
//
//   C = 64, fp16        cf_block64.h  all weights resident in LDS, 64-pixel waves
//   C = 128/256, fp16   cf_wide.h     wave pairs per block, DMA-fed weight buffers
//   C = 512, fp16       cf_wide.h     one wave per block, chunk ring, optional
//                                     hidden groups (fp32 partials + reduction)
//   bf16, other shapes  cf_fused_impl.h
//
// Hidden-split mode (groups > 1): workgroup (tile, g) runs only its range of
// chunks and writes an fp32 partial of the projected output; split_reduce_kernel
// adds the partials in group order plus b2 and the residual.  Batches of at
// most 8 tiles of 128 pixels use the small-batch kernel of cf_small.hip.
#include "cf_block64.h"
#include "cf_wide.h"
#include "cf_fused_impl.h"

#include <mutex>

namespace cf {

namespace fused {
namespace {

// y = x + b2 + sum_g partial[g]  (groups added in increasing order)
template <typename T>
__global__ __launch_bounds__(256) void split_reduce_kernel(const uint16_t *x, uint16_t *y, const float *partial,
                                                           const float *b2, int64_t P, int C, int groups) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;  // one thread per 4 channels
    const int64_t n4 = P * C / 4;
    if (i >= n4)
        return;
    const int64_t e = i * 4;
    const int c = (int)(e % C);
    float4v s = b2 ? *reinterpret_cast<const float4v *>(b2 + c) : float4v{0.f, 0.f, 0.f, 0.f};
    // groups are added in increasing order; eight loads are issued at a time
    int gi = 0;
    for (; gi + 8 <= groups; gi += 8) {
        float4v v[8];
#pragma unroll
        for (int u = 0; u < 8; u++)
            v[u] = *reinterpret_cast<const float4v *>(partial + (size_t)(gi + u) * P * C + e);
#pragma unroll
        for (int u = 0; u < 8; u++)
            s += v[u];
    }
    for (; gi < groups; gi++)
        s += *reinterpret_cast<const float4v *>(partial + (size_t)gi * P * C + e);
    const u32x2 xv = *reinterpret_cast<const u32x2 *>(x + e);
    u32x2 o;
    o[0] = T::pack2(T::lo(xv[0]) + s[0], T::hi(xv[0]) + s[1]);
    o[1] = T::pack2(T::lo(xv[1]) + s[2], T::hi(xv[1]) + s[3]);
    *reinterpret_cast<u32x2 *>(y + e) = o;
}

}  // namespace
}  // namespace fused

using namespace fused;

int device_cu_count() {
    static std::mutex mu;
    static int cached[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64)
        return 256;
    std::lock_guard<std::mutex> lk(mu);
    if (!cached[dev]) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
            n = 256;
        cached[dev] = n;
    }
    return cached[dev];
}

size_t fused_lds_bytes(const Shape &s) {
    if (s.C != 64 && s.C != 128 && s.C != 256 && s.C != 512)
        return 0;
    const int64_t P = (int64_t)s.N * s.H * s.W;
    return lds_bytes_for(s.C, s.k, s.W, s.E, P, 1, false, 1, s.bf16 != 0);
}

hipError_t launch_fused_block(const void *x, void *y, const BlockW &w, const Shape &s, int groups,
                              float *partial, hipStream_t st) {
    FusedArgs a{};
    a.x = (const uint16_t *)x;
    a.y = (uint16_t *)y;
    a.dw_w = (const uint16_t *)w.dw_w;
    a.s0 = w.s0;
    a.b0 = w.b0;
    a.w1 = (const uint16_t *)w.w1;
    a.s1 = w.s1;
    a.b1 = w.b1;
    a.w2 = (const uint16_t *)w.w2;
    a.s2 = w.s2;
    a.b2 = w.b2;
    a.partial = partial;
    a.N = s.N;
    a.H = s.H;
    a.W = s.W;
    a.E = s.E;
    a.P = (uint32_t)((int64_t)s.N * s.H * s.W);
    hipError_t e;
    bool done = false;
    if (groups > 1) {
        e = launch_small_split(x, w, s, groups, partial, st);
        if (e != hipErrorInvalidConfiguration) {
            if (e != hipSuccess)
                return e;
            done = true;
        }
    }
    // a handful of pixels: the slice kernel (no workspace) unless the
    // autotuner chose the tile kernels (CFG_TILE) or the generic one
    if (!done && groups <= 1 && s.cfg == CFG_DEFAULT && slice_applies(s))
        return launch_slice(x, y, w, s, st);
    const bool special = s.cfg != CFG_GENERIC;
    // C = 512 in bf16 has no streaming kernel of its own: the single-group
    // small kernel (one workgroup per 128-pixel tile and 128 output channels,
    // each walking all hidden chunks) replaces the generic kernel, whose tile
    // does not fit the LDS beyond a few image rows.
    if (!done && special && s.C == 512 && s.bf16 && groups <= 1) {
        e = launch_small_split(x, w, s, 1, nullptr, st, y);
        if (e != hipErrorInvalidConfiguration)
            return e;
    }
    if (!done && special && s.C == 64 && !s.bf16 && groups <= 1) {
        switch (s.k) {
        case 1: e = launch_block64_k1(x, y, w, s, st); break;
        case 3: e = launch_block64_k3(x, y, w, s, st); break;
        case 5: e = launch_block64_k5(x, y, w, s, st); break;
        default: e = launch_block64_k7(x, y, w, s, st); break;
        }
        if (e != hipErrorInvalidConfiguration)
            return e;
    }
    if (!done && special && (s.C == 128 || s.C == 256) && !s.bf16 && groups <= 1) {
        e = s.C == 128 ? launch_wide_c128(x, y, w, s, st) : launch_wide_c256(x, y, w, s, st);
        if (e != hipErrorInvalidConfiguration)
            return e;
    }
    if (!done && special && s.C == 512 && !s.bf16) {
        e = launch_wide_c512(x, y, w, s, groups, partial, st);
        if (e != hipErrorInvalidConfiguration) {
            if (e != hipSuccess)
                return e;
            done = true;
        }
    }
    if (!done) {
    switch (s.C * 2 + s.bf16) {
    case 128: e = launch_c64_F16(a, s.k, s.act, groups, st); break;
    case 129: e = launch_c64_BF16(a, s.k, s.act, groups, st); break;
    case 256: e = launch_c128_F16(a, s.k, s.act, groups, st); break;
    case 257: e = launch_c128_BF16(a, s.k, s.act, groups, st); break;
    case 512: e = launch_c256_F16(a, s.k, s.act, groups, st); break;
    case 513: e = launch_c256_BF16(a, s.k, s.act, groups, st); break;
    case 1024: e = launch_c512_F16(a, s.k, s.act, groups, st); break;
    case 1025: e = launch_c512_BF16(a, s.k, s.act, groups, st); break;
    default: return hipErrorInvalidValue;
    }
    }
    if (e != hipSuccess || groups <= 1)
        return e;
    const int64_t n4 = (int64_t)a.P * s.C / 4;
    const int nb = (int)((n4 + 255) / 256);
    if (s.bf16)
        hipLaunchKernelGGL(split_reduce_kernel<BF16>, dim3(nb), dim3(256), 0, st, a.x, a.y, partial, w.b2, a.P, s.C,
                           groups);
    else
        hipLaunchKernelGGL(split_reduce_kernel<F16>, dim3(nb), dim3(256), 0, st, a.x, a.y, partial, w.b2, a.P, s.C,
                           groups);
    return hipGetLastError();
}

bool tile_fits(const Shape &s) {
    const size_t lds = fused_lds_bytes(s);
    if (lds > 0 && lds <= 160 * 1024)
        return true;
    // C = 512 in bf16 runs the single-group small kernel (one 128-pixel tile per
    // workgroup) whenever its halo and D buffer fit
    if (s.C == 512 && s.bf16) {
        const size_t sl = small_split_lds_bytes(s, true);
        return sl > 0 && sl <= 160 * 1024;
    }
    return false;
}

bool cfg_applies(const Shape &s, int cfg) {
    switch (cfg) {
    case CFG_DEFAULT: return true;
    case CFG_GENERIC: return fused_lds_bytes(s) > 0 && fused_lds_bytes(s) <= 160 * 1024;
    case CFG_HALF_TILE: return s.C == 64 && !s.bf16;
    case CFG_TILE: return slice_applies(s) && tile_fits(s);
    default: return false;
    }
}

}  // namespace cf
