// cf_cfs2.hip -- the stride-2 ConvFirst block (Fig. f:convfirst-block (c))
// in one kernel: grouped 3 x 3 conv (group width 8) C -> C with its folded
// norm at the input size, BlurPool (Triangle-3 taps [1, 2, 1] / 4 per
// direction, one pixel of reflect padding, stride 2) of the conv output and
// of the block input, the two maps concatenated (2C channels, conv output
// first) into the expand, activation, project to K, no residual.
//
// Work unit: 16 output pixels of one output row (columns j0 .. j0 + 15), one
// per wave, in a private LDS region:
//  1. the input window, rows 2i - 2 .. 2i + 2 and columns 2j0 - 2 .. 2j0 + 32,
//     zero outside the image (the conv's padding);
//  2. the grouped conv at the full-resolution positions the blur reads --
//     virtual rows 2i - 1 .. 2i + 1 and columns 2j0 - 1 .. 2j0 + 31, each
//     evaluated at its reflected position, so the blur needs no reflection --
//     on the VALU: a lane takes one position and one group of 8 channels,
//     eight outputs of 72 products each as pair products accumulated in
//     fp32 (v_dot2_f32_f16 / _bf16); s0, b0; rounded to the I/O dtype;
//  3. the blur of both maps (fp32, rounded to the I/O dtype) into a 16-pixel
//     tile of 2C channels, zero-padded to a multiple of 32;
//  4. the FFN on v_mfma_f32_16x16x32: expand tiles of 16 hidden channels (A =
//     W1 rows, B = the tile), s1, b1 and the activation in fp32, rounded; two
//     tiles form the B operand of the project with the K order position
//     8q + e <-> hidden 32kk + 4q + e (e < 4) or 32kk + 16 + 4q + e - 4, the
//     lane layout the expand leaves, and the W2 fragments are read in that
//     order; s2, b2; y stored once.
// The input windows of neighbouring units overlap by three columns and the
// conv positions on the unit's border columns are evaluated by both units.
#include "cf_device.h"
#include "cf_kernels.h"

namespace cf {
namespace cfs2 {

constexpr int XR = 5, XC = 35;  // input window: rows 2i-2 .. 2i+2, columns 2j0-2 .. 2j0+32
constexpr int VR = 3, VC = 33;  // conv outputs: virtual rows 2i-1 .. 2i+1, columns 2j0-1 .. 2j0+31
constexpr int UPX = 16;         // output pixels per unit
constexpr int KMAX = 128;       // output channels
constexpr int RMAX = 1024;      // hidden channels

struct Args {
    const uint16_t *x;
    uint16_t *y;
    const uint16_t *gw;  // [3][3][C][8]
    const float *s0, *b0;
    const uint16_t *w1;  // [R][2C]
    const float *s1, *b1;
    const uint16_t *w2;  // [K][R]
    const float *s2, *b2;
    int H, W, Ho, Wo, R, K, act;
    int units, jt;        // units = N * Ho * jt, jt = ceil(Wo / 16)
    int nw;               // waves per workgroup
    uint32_t off_region;  // LDS: the taps at 0, then one region per wave
};

__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c, F16) {
    return __builtin_amdgcn_fdot2(__builtin_bit_cast(half2v, a), __builtin_bit_cast(half2v, b), c, false);
}
__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c, BF16) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a), __builtin_bit_cast(bf16x2, b), c, false);
}

// one pixel of reflect padding (-1 -> 1, n -> n - 2); past that (the padded
// pixels of a unit at the right edge, whose outputs are not stored) the last
// column
__device__ __forceinline__ int refl(int v, int n) {
    if (v < 0)
        return -v;
    if (v == n)
        return n - 2;
    return v > n ? n - 1 : v;
}

__device__ __forceinline__ float act_f(float u, int act) {
    if (act == ACT_RELU)
        return fmaxf(u, 0.0f);
    if (act == ACT_GELU)
        return 0.5f * u * (1.0f + erff(u * 0.70710678118654752f));
    return u;
}

template <typename T, int C>
struct Kern {
    static constexpr int G = C / 8;                            // groups of the conv
    static constexpr uint32_t PP = 2 * C + 16;                 // LDS bytes per window / conv pixel
    static constexpr int C2 = 2 * C, C2P = (C2 + 31) / 32 * 32;
    static constexpr int KS = C2P / 32;                        // expand K steps
    static constexpr uint32_t PZ = 2 * C2P + 16;               // LDS bytes per tile pixel
    static constexpr uint32_t XB = XR * XC * PP, VB = VR * VC * PP, ZB = UPX * PZ;
    static constexpr uint32_t REGION = XB + VB + ZB;

    static __device__ void run(const Args &a, uint8_t *smem) {
        const int tid = threadIdx.x, lane = tid & 63;
        const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
        // the taps [3][3][C][8], once per workgroup
        for (int i = tid; i < 9 * C; i += a.nw * 64)
            *reinterpret_cast<u32x4 *>(smem + (uint32_t)i * 16) =
                *reinterpret_cast<const u32x4 *>(a.gw + (size_t)i * 8);
        __syncthreads();
        const int unit = (int)blockIdx.x * a.nw + wv;
        if (unit >= a.units)
            return;  // (after the workgroup's only barrier)
        const int jt = unit % a.jt, ni = unit / a.jt;
        const int i = ni % a.Ho, n = ni / a.Ho;
        const int j0 = jt * UPX;
        const int H = a.H, W = a.W;
        uint8_t *X = smem + a.off_region + (uint32_t)wv * REGION, *V = X + XB, *Z = V + VB;
        const uint16_t *xn = a.x + (size_t)n * H * W * C;
        const int r0 = 2 * i - 2, c0 = 2 * j0 - 2;

        // 1. the input window (adjacent lanes on adjacent 16-byte pieces)
        for (int t = lane; t < XR * XC * G; t += 64) {
            const int px = t / G, pc = t - px * G, rr = px / XC, cc = px - rr * XC;
            const int gr = r0 + rr, gc = c0 + cc;
            u32x4 v = {0u, 0u, 0u, 0u};
            if (gr >= 0 && gr < H && gc >= 0 && gc < W)
                v = *reinterpret_cast<const u32x4 *>(xn + ((size_t)gr * W + gc) * C + pc * 8);
            *reinterpret_cast<u32x4 *>(X + (uint32_t)px * PP + (uint32_t)pc * 16) = v;
        }

        // 2. the grouped conv at the virtual positions; task = (group, position),
        //    group-major so that the lanes of a pass share the taps they read
        for (int t = lane; t < VR * VC * G; t += 64) {
            const int g = t / (VR * VC), pos = t - g * (VR * VC), vr = pos / VC, vc = pos - vr * VC;
            const int ar = refl(2 * i - 1 + vr, H) - r0, ac = refl(2 * j0 - 1 + vc, W) - c0;  // window coordinates
            float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll 1
            for (int di = 0; di < 3; di++)  // (rolled: the 72 tap reads of an unrolled body would fill the registers)
#pragma unroll
                for (int dj = 0; dj < 3; dj++) {
                    Pack8 xv;
                    xv.u = *reinterpret_cast<const u32x4 *>(X + (uint32_t)((ar + di - 1) * XC + ac + dj - 1) * PP +
                                                            (uint32_t)g * 16);
                    const uint8_t *tp = smem + (uint32_t)(((di * 3 + dj) * C + 8 * g) * 16);
#pragma unroll
                    for (int o = 0; o < 8; o++) {
                        Pack8 w8;
                        w8.u = *reinterpret_cast<const u32x4 *>(tp + o * 16);
#pragma unroll
                        for (int e = 0; e < 4; e++)
                            acc[o] = dot2(xv.w[e], w8.w[e], acc[o], T{});
                    }
                }
            u32x4 out;
#pragma unroll
            for (int e = 0; e < 4; e++) {
                const int c = 8 * g + 2 * e;
                const float sa = a.s0 ? a.s0[c] : 1.0f, sb = a.s0 ? a.s0[c + 1] : 1.0f;
                const float ba = a.b0 ? a.b0[c] : 0.0f, bb = a.b0 ? a.b0[c + 1] : 0.0f;
                out[e] = T::pack2(fmaf(acc[2 * e], sa, ba), fmaf(acc[2 * e + 1], sb, bb));
            }
            *reinterpret_cast<u32x4 *>(V + (uint32_t)pos * PP + (uint32_t)g * 16) = out;
        }

        // 3. BlurPool of the conv output (virtual layout) and of the input
        //    (reflected window positions) into the tile [16][C2P]
        for (int t = lane; t < UPX * (C2P / 4); t += 64) {
            const int px = t / (C2P / 4), c = 4 * (t - px * (C2P / 4));
            float acc[4] = {0.f, 0.f, 0.f, 0.f};
            if (c < C2) {
#pragma unroll
                for (int ta = 0; ta < 3; ta++)
#pragma unroll
                    for (int tb = 0; tb < 3; tb++) {
                        const float wt = (ta == 1 ? 0.5f : 0.25f) * (tb == 1 ? 0.5f : 0.25f);
                        const uint8_t *src;
                        if (c < C) {
                            src = V + (uint32_t)(ta * VC + 2 * px + tb) * PP + (uint32_t)c * 2;
                        } else {
                            const int xr = refl(2 * i + ta - 1, H) - r0, xc = refl(2 * (j0 + px) + tb - 1, W) - c0;
                            src = X + (uint32_t)(xr * XC + xc) * PP + (uint32_t)(c - C) * 2;
                        }
                        const u32x2 v = *reinterpret_cast<const u32x2 *>(src);
                        acc[0] = fmaf(wt, T::lo(v[0]), acc[0]);
                        acc[1] = fmaf(wt, T::hi(v[0]), acc[1]);
                        acc[2] = fmaf(wt, T::lo(v[1]), acc[2]);
                        acc[3] = fmaf(wt, T::hi(v[1]), acc[3]);
                    }
            }
            *reinterpret_cast<u32x2 *>(Z + (uint32_t)px * PZ + (uint32_t)c * 2) =
                u32x2{T::pack2(acc[0], acc[1]), T::pack2(acc[2], acc[3])};
        }

        // 4. the FFN
        const int q = lane >> 4, jl = lane & 15;
        u32x4 zf[KS];
#pragma unroll
        for (int ks = 0; ks < KS; ks++)
            zf[ks] = *reinterpret_cast<const u32x4 *>(Z + (uint32_t)jl * PZ + (uint32_t)(32 * ks + 8 * q) * 2);
        const int R = a.R, OT = (a.K + 15) / 16;  // K % 16 == 8: the last tile's upper half is masked
        float4v acc_o[KMAX / 16];
#pragma unroll
        for (int ot = 0; ot < KMAX / 16; ot++)
            acc_o[ot] = float4v{0.f, 0.f, 0.f, 0.f};
        for (int kk = 0; kk < (R + 31) / 32; kk++) {
            uint32_t hp[4];
#pragma unroll
            for (int t = 0; t < 2; t++) {
                const int h0 = 32 * kk + 16 * t;  // the expand tile's first hidden channel
                float4v u = {0.f, 0.f, 0.f, 0.f};
                if (h0 < R) {  // wave-uniform
                    const uint16_t *wr = a.w1 + (size_t)(h0 + jl) * C2;
#pragma unroll
                    for (int ks = 0; ks < KS; ks++) {
                        const int k = 32 * ks + 8 * q;
                        const u32x4 av = k < C2 ? *reinterpret_cast<const u32x4 *>(wr + k) : u32x4{0u, 0u, 0u, 0u};
                        u = T::mfma(av, zf[ks], u);
                    }
                }
                // lane (q, jl) holds hidden h0 + 4q + e of pixel jl
                const int hh = h0 + 4 * q;
#pragma unroll
                for (int e2 = 0; e2 < 2; e2++) {
                    float v[2];
#pragma unroll
                    for (int s = 0; s < 2; s++) {
                        const int h = hh + 2 * e2 + s;
                        v[s] = 0.0f;
                        if (h0 < R) {
                            const float sc = a.s1 ? a.s1[h] : 1.0f, bi = a.b1 ? a.b1[h] : 0.0f;
                            v[s] = act_f(fmaf(u[2 * e2 + s], sc, bi), a.act);
                        }
                    }
                    hp[2 * t + e2] = T::pack2(v[0], v[1]);
                }
            }
            const u32x4 ub = {hp[0], hp[1], hp[2], hp[3]};
            // W2 rows 16 ot + jl at hidden 32kk + 4q .. + 3 and 32kk + 16 + 4q .. + 3
            const int ha = 32 * kk + 4 * q, hb = ha + 16;
#pragma unroll
            for (int ot = 0; ot < KMAX / 16; ot++) {
                if (ot >= OT)
                    break;
                const bool row = 16 * ot + jl < a.K;
                const uint16_t *wr = a.w2 + (size_t)(row ? 16 * ot + jl : 0) * R;
                const u32x2 pa = row ? *reinterpret_cast<const u32x2 *>(wr + ha) : u32x2{0u, 0u};
                const u32x2 pb = row && hb < R ? *reinterpret_cast<const u32x2 *>(wr + hb) : u32x2{0u, 0u};
                acc_o[ot] = T::mfma(u32x4{pa[0], pa[1], pb[0], pb[1]}, ub, acc_o[ot]);
            }
        }
        // y = s2 * acc + b2: lane (q, jl) holds channels 16 ot + 4q .. + 3 of pixel j0 + jl
        if (j0 + jl < a.Wo) {
            uint16_t *yp = a.y + (((size_t)n * a.Ho + i) * a.Wo + j0 + jl) * a.K;
#pragma unroll
            for (int ot = 0; ot < KMAX / 16; ot++) {
                if (ot >= OT)
                    break;
                const int o = 16 * ot + 4 * q;
                if (o >= a.K)
                    continue;
                float r[4];
#pragma unroll
                for (int e = 0; e < 4; e++)
                    r[e] = fmaf(acc_o[ot][e], a.s2 ? a.s2[o + e] : 1.0f, a.b2 ? a.b2[o + e] : 0.0f);
                *reinterpret_cast<u32x2 *>(yp + o) = u32x2{T::pack2(r[0], r[1]), T::pack2(r[2], r[3])};
            }
        }
    }
};

template <typename T, int C>
__global__ __launch_bounds__(256) void cfs2_kernel(Args a) {
    extern __shared__ __attribute__((aligned(256))) uint8_t smem[];
    Kern<T, C>::run(a, smem);
}

template <int C>
uint32_t region_bytes() {
    return Kern<F16, C>::REGION;
}

inline uint32_t taps_bytes(int C) { return ((uint32_t)(9 * C * 8 * 2) + 255) & ~255u; }

inline uint32_t region_for(int C) {
    switch (C) {
    case 16: return region_bytes<16>();
    case 24: return region_bytes<24>();
    case 32: return region_bytes<32>();
    case 48: return region_bytes<48>();
    case 64: return region_bytes<64>();
    default: return 0;
    }
}

// waves per workgroup: as many as four regions fit beside the taps
inline int waves_for(int C) {
    const uint32_t r = region_for(C);
    if (!r)
        return 0;
    int nw = (int)((160u * 1024u - taps_bytes(C)) / r);
    return nw > 4 ? 4 : nw;
}

template <typename T, int C>
hipError_t launch_t(const Args &a, size_t lds, int grid, hipStream_t st) {
    auto kf = cfs2_kernel<T, C>;
    hipError_t e = allow_full_lds((const void *)kf);
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(kf, dim3(grid), dim3(64 * a.nw), lds, st, a);
    return hipGetLastError();
}

template <typename T>
hipError_t launch_c(const Args &a, int C, size_t lds, int grid, hipStream_t st) {
    switch (C) {
    case 16: return launch_t<T, 16>(a, lds, grid, st);
    case 24: return launch_t<T, 24>(a, lds, grid, st);
    case 32: return launch_t<T, 32>(a, lds, grid, st);
    case 48: return launch_t<T, 48>(a, lds, grid, st);
    case 64: return launch_t<T, 64>(a, lds, grid, st);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace cfs2

bool convfirst_s2_supported(int H, int W, int C, int R, int K) {
    return H >= 2 && W >= 2 && cfs2::waves_for(C) >= 1 && R >= 16 && R % 16 == 0 && R <= cfs2::RMAX &&
           K >= 8 && K % 8 == 0 && K <= cfs2::KMAX;
}

hipError_t launch_convfirst_s2(const void *x, void *y, const BlockW &w, int N, int H, int W, int C, int R, int K,
                               int bf16, int act, hipStream_t st) {
    if (!convfirst_s2_supported(H, W, C, R, K))
        return hipErrorInvalidConfiguration;
    cfs2::Args a{};
    a.x = (const uint16_t *)x;
    a.y = (uint16_t *)y;
    a.gw = (const uint16_t *)w.dw_w;
    a.s0 = w.s0;
    a.b0 = w.b0;
    a.w1 = (const uint16_t *)w.w1;
    a.s1 = w.s1;
    a.b1 = w.b1;
    a.w2 = (const uint16_t *)w.w2;
    a.s2 = w.s2;
    a.b2 = w.b2;
    a.H = H;
    a.W = W;
    a.Ho = (H + 1) / 2;
    a.Wo = (W + 1) / 2;
    a.R = R;
    a.K = K;
    a.act = act;
    a.jt = (a.Wo + cfs2::UPX - 1) / cfs2::UPX;
    const int64_t units = (int64_t)N * a.Ho * a.jt;
    if (units <= 0)
        return hipSuccess;
    if (units > (int64_t)1 << 30)
        return hipErrorInvalidValue;
    a.units = (int)units;
    a.nw = cfs2::waves_for(C);
    a.off_region = cfs2::taps_bytes(C);
    const size_t lds = a.off_region + (size_t)a.nw * cfs2::region_for(C);
    const int grid = (a.units + a.nw - 1) / a.nw;
    return bf16 ? cfs2::launch_c<BF16>(a, C, lds, grid, st) : cfs2::launch_c<F16>(a, C, lds, grid, st);
}

}  // namespace cf
