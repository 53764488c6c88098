// cf_stem.hip -- the network's stem (App. A of Lavin, arXiv:2404.03617: a
// 3 x 3 convolution with stride 2 from the image's 3 channels to the first
// stage's 16, 24 or 32; ReLU, caption of Fig. f:convfirstnet) fused into the
// first ConvFirst block, as the appendix proposes: the grouped-block kernel
// computes each block's halo of stem output from the image (cf_gblock.h,
// STEM), so the stem output never reaches memory.  The stem alone
// (stem_kernel) writes its output, for the unfused schedule.
#include "cf_gblock.h"

namespace cf {

namespace {

// y[p][c] = ReLU(s[c] * conv(x)[p][c] + b[c]) for 16-pixel tiles of the
// flattened output, two v_mfma_f32_16x16x32 per tile and 16 channels in the
// K order of the fused kernel.  C = 24 runs two channel tiles, the second
// with zero weights beyond channel 23 and stores of its first 8 channels.
template <typename T, int C>
__global__ __launch_bounds__(256) void stem_kernel(const uint16_t *x, uint16_t *y, const uint16_t *w, const float *s,
                                                   const float *b, int N, int Hin, int Win, int Hs, int Ws) {
    constexpr int SMT = (C + 15) / 16;
    const int lane = threadIdx.x & 63, q = lane >> 4, jl = lane & 15;
    u32x4 sa[SMT][2];
    float4v sc[SMT], bi[SMT];
#pragma unroll
    for (int mt = 0; mt < SMT; mt++) {
        const bool oc = 16 * mt + jl < C;
        sa[mt][0] = oc ? gblk::stem_afrag_px(w, 16 * mt + jl, 0, q) : u32x4{0u, 0u, 0u, 0u};
        sa[mt][1] = oc ? gblk::stem_afrag_px(w, 16 * mt + jl, 1, q) : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
        for (int e = 0; e < 4; e++) {
            const int c = 16 * mt + 4 * q + e;
            sc[mt][e] = s && c < C ? s[c] : 1.0f;
            bi[mt][e] = b && c < C ? b[c] : 0.0f;
        }
    }
    const int64_t P = (int64_t)N * Hs * Ws;
    const int64_t tiles = (P + 15) / 16;
    const int64_t nw = (int64_t)gridDim.x * 4;
    for (int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); t < tiles; t += nw) {
        const int64_t p = 16 * t + jl;
        const bool in = p < P;
        const int64_t pp = in ? p : 0;
        const int n = (int)(pp / ((int64_t)Hs * Ws));
        const int rem = (int)(pp - (int64_t)n * Hs * Ws);
        const int sr = rem / Ws, scol = rem - sr * Ws;
        const uint16_t *img = x + (size_t)n * Hin * Win * 3;
        const u32x4 b0 = gblk::stem_bfrag_px(img, Hin, Win, sr, scol, 0, q, in);
        const u32x4 b1 = gblk::stem_bfrag_px(img, Hin, Win, sr, scol, 1, q, in);
#pragma unroll
        for (int mt = 0; mt < SMT; mt++) {
            float4v acc = T::mfma(sa[mt][0], b0, float4v{0.f, 0.f, 0.f, 0.f});
            acc = T::mfma(sa[mt][1], b1, acc);
            float u[4];
#pragma unroll
            for (int e = 0; e < 4; e++)
                u[e] = fmaxf(fmaf(acc[e], sc[mt][e], bi[mt][e]), 0.0f);
            if (in && 16 * mt + 4 * q < C)
                *reinterpret_cast<u32x2 *>(y + (size_t)p * C + 16 * mt + 4 * q) =
                    u32x2{T::pack2(u[0], u[1]), T::pack2(u[2], u[3])};
        }
    }
}

}  // namespace

hipError_t launch_stem_gblock(const StemW &stem, void *y, const GBlockW &w, const Shape &s, hipStream_t st) {
    switch (s.C) {
    case 16: return gblk::launch_c<16, true>(nullptr, y, w, s, st, &stem);
    case 32: return gblk::launch_c<32, true>(nullptr, y, w, s, st, &stem);
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_stem(const StemW &stem, void *y, int N, int C, int bf16, hipStream_t st) {
    const int Hs = (stem.Hin + 1) / 2, Ws = (stem.Win + 1) / 2;
    const int64_t tiles = ((int64_t)N * Hs * Ws + 15) / 16;
    const int64_t cap = (int64_t)device_cu_count() * 16;
    const int grid = (int)std::max<int64_t>(1, std::min<int64_t>((tiles + 3) / 4, cap));
    const uint16_t *x = (const uint16_t *)stem.x, *w = (const uint16_t *)stem.w;
    uint16_t *yy = (uint16_t *)y;
#define CF_STEM_LAUNCH(TT, CC)                                                                                   \
    hipLaunchKernelGGL((stem_kernel<TT, CC>), dim3(grid), dim3(256), 0, st, x, yy, w, stem.s, stem.b, N, stem.Hin, \
                       stem.Win, Hs, Ws)
    switch (C * 2 + (bf16 ? 1 : 0)) {
    case 32: CF_STEM_LAUNCH(F16, 16); break;
    case 33: CF_STEM_LAUNCH(BF16, 16); break;
    case 48: CF_STEM_LAUNCH(F16, 24); break;
    case 49: CF_STEM_LAUNCH(BF16, 24); break;
    case 64: CF_STEM_LAUNCH(F16, 32); break;
    case 65: CF_STEM_LAUNCH(BF16, 32); break;
    default: return hipErrorInvalidValue;
    }
#undef CF_STEM_LAUNCH
    return hipGetLastError();
}

}  // namespace cf
