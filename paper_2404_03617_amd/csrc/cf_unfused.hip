// cf_unfused.hip -- layer-by-layer kernels for gfx950: the comparison path
// of Fig. f:convfirst-tensor-machine (a) (depth-wise conv, expand GEMM with
// activation, project GEMM with residual, every intermediate through HBM) and
// the 2x2 stride-2 down-sampling conv between stages.
//
// GEMM shape used throughout ("TN"): Out[p][o] = epi( sum_k A[p][k] * B[o][k] )
// with both operands K-contiguous.  Computed transposed on MFMA 16x16x32
// (A operand = B rows, B operand = A rows) so that each lane ends up with 4
// consecutive output channels of one pixel: an 8-byte NHWC store.
#include "cf_device.h"
#include "cf_kernels.h"

namespace cf {

namespace {

// ---------------------------------------------------------------------------
// Depth-wise k x k conv, NHWC, zero padding k/2: one thread = 8 channels of
// one pixel, fp32 accumulation, d = s0 * acc + b0.  The thread index is split
// into (pixel, channel group) and the pixel into (n, h, w) by 32-bit
// multiply-high division when N*H*W*C/8 < 2^31 (64-bit division otherwise).
struct DwDiv {
    FastDiv c8, w, h;
    int small;  // N*H*W*C/8 < 2^31
};

template <typename T, int KS>
__global__ __launch_bounds__(256) void dw_kernel(const uint16_t *x, uint16_t *d, const uint16_t *w, const float *s0,
                                                 const float *b0, int N, int H, int W, int C, DwDiv dv) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int c8 = C / 8;
    const int64_t total = (int64_t)N * H * W * c8;
    if (t >= total)
        return;
    int q8, wc, h;
    int64_t pix, n;
    if (dv.small) {
        const uint32_t tt = (uint32_t)t, px = fdiv(tt, dv.c8), nh = fdiv(px, dv.w), nn = fdiv(nh, dv.h);
        q8 = (int)(tt - px * (uint32_t)c8);
        wc = (int)(px - nh * (uint32_t)W);
        h = (int)(nh - nn * (uint32_t)H);
        pix = px;
        n = nn;
    } else {
        q8 = (int)(t % c8);
        pix = t / c8;
        wc = (int)(pix % W);
        const int64_t nh = pix / W;
        h = (int)(nh % H);
        n = nh / H;
    }
    const int c0 = q8 * 8;
    constexpr int PAD = KS / 2;
    float acc[8];
#pragma unroll
    for (int e = 0; e < 8; e++)
        acc[e] = 0.f;
#pragma unroll
    for (int i = 0; i < KS; i++) {
        const int hh = h + i - PAD;
        if (hh < 0 || hh >= H)
            continue;
#pragma unroll
        for (int j = 0; j < KS; j++) {
            const int ww = wc + j - PAD;
            if (ww < 0 || ww >= W)
                continue;
            Pack8 xv, wv;
            xv.u = *reinterpret_cast<const u32x4 *>(x + (((n * H + hh) * W + ww) * C + c0));
            wv.u = *reinterpret_cast<const u32x4 *>(w + ((size_t)(i * KS + j) * C + c0));
#pragma unroll
            for (int q = 0; q < 4; q++) {
                acc[2 * q] = fmaf(T::lo(xv.w[q]), T::lo(wv.w[q]), acc[2 * q]);
                acc[2 * q + 1] = fmaf(T::hi(xv.w[q]), T::hi(wv.w[q]), acc[2 * q + 1]);
            }
        }
    }
    u32x4 o;
#pragma unroll
    for (int q = 0; q < 4; q++) {
        const int c = c0 + 2 * q;
        const float sa = s0 ? s0[c] : 1.f, sb = s0 ? s0[c + 1] : 1.f;
        const float ba = b0 ? b0[c] : 0.f, bb = b0 ? b0[c + 1] : 0.f;
        o[q] = T::pack2(fmaf(acc[2 * q], sa, ba), fmaf(acc[2 * q + 1], sb, bb));
    }
    *reinterpret_cast<u32x4 *>(d + pix * C + c0) = o;
}

// ---------------------------------------------------------------------------
// Tiled MFMA GEMM.  Block tile BM pixels x BN outputs x GK of K, 4 waves as
// 2 x 2, each wave (BM/2) x (BN/2).  Operand tiles go global -> registers ->
// LDS with a padded row stride against bank conflicts; LDS is double
// buffered and the register copies run two K steps ahead, so two global
// round trips are in flight while a step computes.
enum { EPI_EXPAND = 0, EPI_PROJECT = 1, EPI_AFFINE = 2 };
enum { A_PLAIN = 0, A_SPACE_TO_DEPTH = 1 };

struct GemmArgs {
    const uint16_t *a;   // A rows (pixels), K contiguous; or x for space-to-depth
    const uint16_t *b;   // B rows (outputs), K contiguous
    uint16_t *out;       // [P][NO]
    const float *scale;  // [NO] or null
    const float *bias;   // [NO] or null
    const uint16_t *res; // residual [P][NO] (project) or null
    int64_t P;
    int K, NO;
    int act;
    // space-to-depth view: x is [N][2*Ho][2*Wo][Cin], row p = (n, i, j), K = 4*Cin
    // (P < 2^31: 32-bit multiply-high division by Wo, Ho and Cin)
    int Ho, Wo, Cin;
    FastDiv divWo, divHo, divCin;
};


// Start of A row p (its K = 0 element): for the space-to-depth view,
// k = (a*2 + b)*Cin + c reads x[n][2i+a][2j+b][c], and row p = (n, i, j)
// starts at x[n][2i][2j][0]; a K step of GK never crosses a (a, b) boundary
// (Cin is a multiple of GK), so a load is row start + tap offset + c.
template <int AMODE>
__device__ __forceinline__ const uint16_t *a_row_start(const GemmArgs &g, int64_t p) {
    if constexpr (AMODE == A_PLAIN) {
        return g.a + p * g.K;
    } else {
        const uint32_t pp = (uint32_t)p, ni = fdiv(pp, g.divWo), j = pp - ni * (uint32_t)g.Wo;
        const uint32_t n = fdiv(ni, g.divHo), i = ni - n * (uint32_t)g.Ho;
        const size_t W = 2 * (size_t)g.Wo;
        return g.a + (((size_t)n * 2 * g.Ho + 2 * i) * W + 2 * j) * g.Cin;
    }
}
// offset of element k from the row start
template <int AMODE>
__device__ __forceinline__ int64_t a_col_off(const GemmArgs &g, int k) {
    if constexpr (AMODE == A_PLAIN) {
        return k;
    } else {
        const int ab = (int)fdiv((uint32_t)k, g.divCin), c = k - ab * g.Cin;
        return ((int64_t)(ab >> 1) * 2 * g.Wo + (ab & 1)) * g.Cin + c;
    }
}

template <typename T, int BM, int BN, int GK, int EPI, int AMODE>
__global__ __launch_bounds__(256) void gemm_kernel(GemmArgs g) {
    constexpr int LDS_STRIDE = GK + 8;  // halves per LDS row (8 halves of padding)
    constexpr int WM = BM / 2, WN = BN / 2;  // per-wave tile (pixels x outputs)
    constexpr int FM = WM / 16, FN = WN / 16;
    constexpr int A_PIECES = BM * GK / 8 / 256;  // 16-byte pieces per thread
    constexpr int B_PIECES = BN * GK / 8 / 256;
    __shared__ __attribute__((aligned(16))) uint16_t sa[2][BM * LDS_STRIDE];
    __shared__ __attribute__((aligned(16))) uint16_t sb[2][BN * LDS_STRIDE];

    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int wm = wv >> 1, wn = wv & 1;
    const int64_t p0 = (int64_t)blockIdx.x * BM;
    const int o0 = blockIdx.y * BN;

    float4v acc[FN][FM];
#pragma unroll
    for (int i = 0; i < FN; i++)
#pragma unroll
        for (int j = 0; j < FM; j++)
            acc[i][j] = float4v{0.f, 0.f, 0.f, 0.f};

    // this thread's A rows, decomposed once
    const uint16_t *arow[A_PIECES];
    bool aok[A_PIECES];
#pragma unroll
    for (int q = 0; q < A_PIECES; q++) {
        const int64_t p = p0 + (q * 256 + tid) / (GK / 8);
        aok[q] = p < g.P;
        arow[q] = a_row_start<AMODE>(g, aok[q] ? p : 0);
    }
    u32x4 ra[A_PIECES], rbv[B_PIECES];
    auto load = [&](int k0) {
        const int64_t koff = a_col_off<AMODE>(g, k0);
#pragma unroll
        for (int q = 0; q < A_PIECES; q++) {
            const int c8 = (q * 256 + tid) % (GK / 8);
            ra[q] = aok[q] ? *reinterpret_cast<const u32x4 *>(arow[q] + koff + c8 * 8) : u32x4{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int q = 0; q < B_PIECES; q++) {
            const int pc = q * 256 + tid;
            const int r = pc / (GK / 8), c8 = pc % (GK / 8);
            rbv[q] = *reinterpret_cast<const u32x4 *>(g.b + (size_t)(o0 + r) * g.K + k0 + c8 * 8);
        }
    };
    auto store = [&](int buf) {
#pragma unroll
        for (int q = 0; q < A_PIECES; q++) {
            const int pc = q * 256 + tid;
            const int r = pc / (GK / 8), c8 = pc % (GK / 8);
            *reinterpret_cast<u32x4 *>(&sa[buf][r * LDS_STRIDE + c8 * 8]) = ra[q];
        }
#pragma unroll
        for (int q = 0; q < B_PIECES; q++) {
            const int pc = q * 256 + tid;
            const int r = pc / (GK / 8), c8 = pc % (GK / 8);
            *reinterpret_cast<u32x4 *>(&sb[buf][r * LDS_STRIDE + c8 * 8]) = rbv[q];
        }
    };

    const int nk = g.K / GK;
    auto compute = [&](int buf) {
#pragma unroll
        for (int ks = 0; ks < GK / 32; ks++) {
            u32x4 fa[FN], fb[FM];
#pragma unroll
            for (int i = 0; i < FN; i++)
                fa[i] = *reinterpret_cast<const u32x4 *>(
                    &sb[buf][(wn * WN + i * 16 + (lane & 15)) * LDS_STRIDE + 32 * ks + 8 * (lane >> 4)]);
#pragma unroll
            for (int j = 0; j < FM; j++)
                fb[j] = *reinterpret_cast<const u32x4 *>(
                    &sa[buf][(wm * WM + j * 16 + (lane & 15)) * LDS_STRIDE + 32 * ks + 8 * (lane >> 4)]);
#pragma unroll
            for (int i = 0; i < FN; i++)
#pragma unroll
                for (int j = 0; j < FM; j++)
                    acc[i][j] = T::mfma(fa[i], fb[j], acc[i][j]);
        }
    };
    // two register sets: set (kt & 1) holds K step kt + 2 once its loads land
    u32x4 ra2[A_PIECES], rb2[B_PIECES];
    load(0);
    store(0);
    if (nk > 1)
        load(GK);
#pragma unroll
    for (int q = 0; q < A_PIECES; q++)
        ra2[q] = ra[q];
#pragma unroll
    for (int q = 0; q < B_PIECES; q++)
        rb2[q] = rbv[q];
    // ra2/rb2: step 1 (if any); ra/rbv: free
    for (int kt = 0; kt < nk; kt++) {
        __syncthreads();
        const int buf = kt & 1;
        if (kt + 2 < nk)
            load((kt + 2) * GK);  // into ra/rbv
        compute(buf);
        if (kt + 1 < nk) {
            // step kt + 1 (in ra2/rb2) goes to the other LDS buffer
#pragma unroll
            for (int q = 0; q < A_PIECES; q++) {
                const int pc = q * 256 + tid;
                const int r = pc / (GK / 8), c8 = pc % (GK / 8);
                *reinterpret_cast<u32x4 *>(&sa[buf ^ 1][r * LDS_STRIDE + c8 * 8]) = ra2[q];
            }
#pragma unroll
            for (int q = 0; q < B_PIECES; q++) {
                const int pc = q * 256 + tid;
                const int r = pc / (GK / 8), c8 = pc % (GK / 8);
                *reinterpret_cast<u32x4 *>(&sb[buf ^ 1][r * LDS_STRIDE + c8 * 8]) = rb2[q];
            }
        }
        // the loads of step kt + 2 become the next step's pending set
#pragma unroll
        for (int q = 0; q < A_PIECES; q++)
            ra2[q] = ra[q];
#pragma unroll
        for (int q = 0; q < B_PIECES; q++)
            rb2[q] = rbv[q];
    }

    // epilogue: lane holds outputs o0 + wn*WN + i*16 + 4*(lane>>4) + e, pixel p0 + wm*WM + j*16 + (lane&15)
#pragma unroll
    for (int j = 0; j < FM; j++) {
        const int64_t p = p0 + wm * WM + j * 16 + (lane & 15);
        if (p >= g.P)
            continue;
#pragma unroll
        for (int i = 0; i < FN; i++) {
            const int o = o0 + wn * WN + i * 16 + 4 * (lane >> 4);
            float v[4];
#pragma unroll
            for (int e = 0; e < 4; e++) {
                const float s = g.scale ? g.scale[o + e] : 1.f;
                const float bb = g.bias ? g.bias[o + e] : 0.f;
                v[e] = fmaf(acc[i][j][e], s, bb);
            }
            if constexpr (EPI == EPI_EXPAND) {
#pragma unroll
                for (int e = 0; e < 4; e++) {
                    if (g.act == ACT_GELU)
                        v[e] = gelu_f32(v[e]);
                    else if (g.act == ACT_RELU)
                        v[e] = fmaxf(v[e], 0.f);
                }
            } else if constexpr (EPI == EPI_PROJECT) {
                const u32x2 xr = *reinterpret_cast<const u32x2 *>(g.res + p * g.NO + o);
                v[0] += T::lo(xr[0]);
                v[1] += T::hi(xr[0]);
                v[2] += T::lo(xr[1]);
                v[3] += T::hi(xr[1]);
            }
            u32x2 ov;
            ov[0] = T::pack2(v[0], v[1]);
            ov[1] = T::pack2(v[2], v[3]);
            *reinterpret_cast<u32x2 *>(g.out + p * g.NO + o) = ov;
        }
    }
}

template <typename T, int GK, int EPI, int AMODE>
hipError_t gemm_k(const GemmArgs &g, hipStream_t st) {
    // BN must divide NO; all NO used here are multiples of 64.  Where 128 x 128
    // tiles would leave compute units short of work, 64-pixel tiles (the
    // small weight operand is re-read, not the activations).
    const int64_t tiles128 = ((g.P + 127) / 128) * (g.NO / 128);
    if (g.NO % 128 == 0 && tiles128 >= 2 * device_cu_count()) {
        dim3 grid((unsigned)((g.P + 127) / 128), g.NO / 128);
        hipLaunchKernelGGL((gemm_kernel<T, 128, 128, GK, EPI, AMODE>), grid, dim3(256), 0, st, g);
    } else if (g.NO % 128 == 0) {
        dim3 grid((unsigned)((g.P + 63) / 64), g.NO / 128);
        hipLaunchKernelGGL((gemm_kernel<T, 64, 128, GK, EPI, AMODE>), grid, dim3(256), 0, st, g);
    } else {
        dim3 grid((unsigned)((g.P + 127) / 128), g.NO / 64);
        hipLaunchKernelGGL((gemm_kernel<T, 128, 64, GK, EPI, AMODE>), grid, dim3(256), 0, st, g);
    }
    return hipGetLastError();
}

template <typename T, int EPI, int AMODE>
hipError_t gemm(const GemmArgs &g, hipStream_t st) {
    if constexpr (AMODE == A_PLAIN) {
        // layer-by-layer GEMMs (large P): 128-pixel tiles, K steps of 32
        if (g.NO % 128 == 0) {
            dim3 grid((unsigned)((g.P + 127) / 128), g.NO / 128);
            hipLaunchKernelGGL((gemm_kernel<T, 128, 128, 32, EPI, AMODE>), grid, dim3(256), 0, st, g);
        } else {
            dim3 grid((unsigned)((g.P + 127) / 128), g.NO / 64);
            hipLaunchKernelGGL((gemm_kernel<T, 128, 64, 32, EPI, AMODE>), grid, dim3(256), 0, st, g);
        }
        return hipGetLastError();
    } else {
        // down-sampling: K steps of 64 where Cin allows it
        return g.Cin % 64 == 0 ? gemm_k<T, 64, EPI, AMODE>(g, st) : gemm_k<T, 32, EPI, AMODE>(g, st);
    }
}

template <typename T>
hipError_t dw(const void *x, void *d, const BlockW &w, const Shape &s, hipStream_t st) {
    const int64_t total = (int64_t)s.N * s.H * s.W * (s.C / 8);
    const unsigned nb = (unsigned)((total + 255) / 256);
    const uint16_t *xx = (const uint16_t *)x;
    uint16_t *dd = (uint16_t *)d;
    const uint16_t *ww = (const uint16_t *)w.dw_w;
    DwDiv dv;
    dv.c8 = make_fastdiv((uint32_t)(s.C / 8));
    dv.w = make_fastdiv((uint32_t)s.W);
    dv.h = make_fastdiv((uint32_t)s.H);
    dv.small = total < ((int64_t)1 << 31) ? 1 : 0;
    switch (s.k) {
    case 1: hipLaunchKernelGGL((dw_kernel<T, 1>), dim3(nb), dim3(256), 0, st, xx, dd, ww, w.s0, w.b0, s.N, s.H, s.W, s.C, dv); break;
    case 3: hipLaunchKernelGGL((dw_kernel<T, 3>), dim3(nb), dim3(256), 0, st, xx, dd, ww, w.s0, w.b0, s.N, s.H, s.W, s.C, dv); break;
    case 5: hipLaunchKernelGGL((dw_kernel<T, 5>), dim3(nb), dim3(256), 0, st, xx, dd, ww, w.s0, w.b0, s.N, s.H, s.W, s.C, dv); break;
    case 7: hipLaunchKernelGGL((dw_kernel<T, 7>), dim3(nb), dim3(256), 0, st, xx, dd, ww, w.s0, w.b0, s.N, s.H, s.W, s.C, dv); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <typename T>
hipError_t unfused(const void *x, void *y, void *d, void *h, const BlockW &w, const Shape &s, hipStream_t st) {
    hipError_t e = dw<T>(x, d, w, s, st);
    if (e != hipSuccess)
        return e;
    const int64_t P = (int64_t)s.N * s.H * s.W;
    const int EC = s.E * s.C;
    GemmArgs g1{};
    g1.a = (const uint16_t *)d;
    g1.b = (const uint16_t *)w.w1;
    g1.out = (uint16_t *)h;
    g1.scale = w.s1;
    g1.bias = w.b1;
    g1.P = P;
    g1.K = s.C;
    g1.NO = EC;
    g1.act = s.act;
    e = gemm<T, EPI_EXPAND, A_PLAIN>(g1, st);
    if (e != hipSuccess)
        return e;
    GemmArgs g2{};
    g2.a = (const uint16_t *)h;
    g2.b = (const uint16_t *)w.w2;
    g2.out = (uint16_t *)y;
    g2.scale = w.s2;
    g2.bias = w.b2;
    g2.res = (const uint16_t *)x;
    g2.P = P;
    g2.K = EC;
    g2.NO = s.C;
    return gemm<T, EPI_PROJECT, A_PLAIN>(g2, st);
}

}  // namespace

hipError_t launch_depthwise(const void *x, void *d, const BlockW &w, const Shape &s, hipStream_t st) {
    return s.bf16 ? dw<BF16>(x, d, w, s, st) : dw<F16>(x, d, w, s, st);
}

hipError_t launch_unfused_block(const void *x, void *y, void *d, void *h, const BlockW &w, const Shape &s,
                                hipStream_t st) {
    return s.bf16 ? unfused<BF16>(x, y, d, h, w, s, st) : unfused<F16>(x, y, d, h, w, s, st);
}

hipError_t launch_downsample(const void *x, void *y, const void *wd, const float *sd, const float *bd, int N, int H,
                             int W, int Cin, int Cout, int bf16, hipStream_t st) {
    GemmArgs g{};
    g.a = (const uint16_t *)x;
    g.b = (const uint16_t *)wd;
    g.out = (uint16_t *)y;
    g.scale = sd;
    g.bias = bd;
    g.Ho = H / 2;
    g.Wo = W / 2;
    g.Cin = Cin;
    g.P = (int64_t)N * g.Ho * g.Wo;
    g.K = 4 * Cin;
    g.NO = Cout;
    if (g.P >= ((int64_t)1 << 31))
        return hipErrorInvalidValue;
    g.divWo = make_fastdiv((uint32_t)g.Wo);
    g.divHo = make_fastdiv((uint32_t)g.Ho);
    g.divCin = make_fastdiv((uint32_t)Cin);
    return bf16 ? gemm<BF16, EPI_AFFINE, A_SPACE_TO_DEPTH>(g, st) : gemm<F16, EPI_AFFINE, A_SPACE_TO_DEPTH>(g, st);
}

}  // namespace cf
