// cf_libgemm.hip -- a ConvFirst block (Sec. 5.2: depth-wise conv, expand,
// activation, project, residual) as five launches whose two pointwise layers
// are plain hipBLASLt GEMMs, for wide blocks over many pixels: at C = 512 and
// N x 7 x 7 pixels (the last stage of the four-stage stack) the two GEMMs
// (P x 512 x 2048 each way) carry all but 1% of the operations and the
// library's GEMM kernels run them at several times the rate of the fused
// kernel, whose 2048 hidden channels per pixel must stream their weights
// through LDS.  The hidden tensor goes through HBM (the layer-by-layer
// schedule of Sec. 5.2; 4 bytes per hidden element for P x 2048 elements).
//
// Launches, all on the caller's stream:
//   1. depth-wise k x k conv, s0, b0 -> D [P][C]            (small images and
//      k = 3: one image slice per workgroup in LDS; else cf_unfused.hip)
//   2. Hraw = D W1^T                  -> H [P][E C]          (hipBLASLt, fp32 accumulate)
//   3. H = act(s1 Hraw + b1): in the GEMM's epilogue (alpha vector, bias,
//      the library's GELU / ReLU) when s1 and b1 are given and the library
//      has such an algorithm; else in place, s1, b1 in fp32, GELU as the
//      fused fp16 kernels evaluate it (packed fp16 on u / 4)
//   4. T = H W2^T                     -> T [P][C]            (hipBLASLt)
//   5. y = s2 T + b2 + x                                      fp32 math, rounded
//      (4 and 5 as one GEMM with the alpha vector s2, x as the C operand
//      and the bias b2 in its epilogue, when s2 and b2 are given)
// The GEMMs get no library workspace, so the library picks no algorithm that
// clears memory on the stream (safe inside a captured graph).  Rounding
// points differ from the fused kernels (T, and Hraw without the epilogue,
// are rounded to fp16 before their scale and bias); the results stay within
// the block tolerance.
#include <hipblaslt/hipblaslt.h>

#include <mutex>

#include "cf_device.h"
#include "cf_kernels.h"

namespace cf {
namespace lgm {

constexpr int MAX_DEV = 16;
constexpr int MAX_SHAPES = 16;

// epilogues: none, or the expand's s1 (a per-row alpha vector), b1 (bias)
// and activation fused into the GEMM
enum { EPI_NONE = 0, EPI_VEC = 1, EPI_VEC_BIAS = 2 };

struct Plan {
    int dev = -1, m = 0, n = 0, k = 0;
    int epi = EPI_NONE, act = 0;
    bool valid = false;  // false: the library had no algorithm (not asked again)
    hipblasLtMatmulDesc_t op = nullptr;
    hipblasLtMatrixLayout_t la = nullptr, lb = nullptr, lc = nullptr;
    hipblasLtMatmulAlgo_t algo{};
};

std::mutex g_mu;
hipblasLtHandle_t g_handle[MAX_DEV] = {};
Plan g_plans[MAX_SHAPES];
int g_nplans = 0;

// D [n][m] (row-major, fp16) = B [n][k] . A [m][k]^T: in the library's
// column-major terms D (m x n) = op(A) (m x k, A stored k x m, transposed)
// times B (k x n).  Plans (descriptors and the heuristic's first algorithm)
// are cached per device and shape; the caller holds g_mu.  With create
// false only an existing plan is returned.
hipError_t plan_for(int dev, int m, int n, int k, const Plan **out, bool create = true, int epi = EPI_NONE,
                    int act = 0) {
    for (int i = 0; i < g_nplans; i++)
        if (g_plans[i].dev == dev && g_plans[i].m == m && g_plans[i].n == n && g_plans[i].k == k &&
            g_plans[i].epi == epi && g_plans[i].act == act) {
            *out = &g_plans[i];
            return g_plans[i].valid ? hipSuccess : hipErrorNotSupported;
        }
    if (!create || g_nplans == MAX_SHAPES)
        return hipErrorNotSupported;
    if (!g_handle[dev] && hipblasLtCreate(&g_handle[dev]) != HIPBLAS_STATUS_SUCCESS)
        return hipErrorNotSupported;
    Plan p;
    p.dev = dev;
    p.m = m;
    p.n = n;
    p.k = k;
    p.epi = epi;
    p.act = act;
    const hipblasOperation_t ta = HIPBLAS_OP_T, tb = HIPBLAS_OP_N;
    uint32_t ep = HIPBLASLT_EPILOGUE_DEFAULT;
    if (epi != EPI_NONE) {
        const bool bias = epi == EPI_VEC_BIAS;
        ep = act == ACT_GELU   ? (bias ? HIPBLASLT_EPILOGUE_GELU_BIAS : HIPBLASLT_EPILOGUE_GELU)
             : act == ACT_RELU ? (bias ? HIPBLASLT_EPILOGUE_RELU_BIAS : HIPBLASLT_EPILOGUE_RELU)
                               : (bias ? HIPBLASLT_EPILOGUE_BIAS : HIPBLASLT_EPILOGUE_DEFAULT);
    }
    const int32_t pmode = HIPBLASLT_POINTER_MODE_ALPHA_DEVICE_VECTOR_BETA_HOST;
    const int32_t btype = HIP_R_32F;
    hipblasLtMatmulPreference_t pref = nullptr;
    const uint64_t no_ws = 0;
    hipblasLtMatmulHeuristicResult_t res[1];
    int nres = 0;
    bool ok = hipblasLtMatmulDescCreate(&p.op, HIPBLAS_COMPUTE_32F, HIP_R_32F) == HIPBLAS_STATUS_SUCCESS &&
              hipblasLtMatmulDescSetAttribute(p.op, HIPBLASLT_MATMUL_DESC_TRANSA, &ta, sizeof(ta)) ==
                  HIPBLAS_STATUS_SUCCESS &&
              hipblasLtMatmulDescSetAttribute(p.op, HIPBLASLT_MATMUL_DESC_TRANSB, &tb, sizeof(tb)) ==
                  HIPBLAS_STATUS_SUCCESS &&
              hipblasLtMatmulDescSetAttribute(p.op, HIPBLASLT_MATMUL_DESC_EPILOGUE, &ep, sizeof(ep)) ==
                  HIPBLAS_STATUS_SUCCESS &&
              (epi == EPI_NONE || hipblasLtMatmulDescSetAttribute(p.op, HIPBLASLT_MATMUL_DESC_POINTER_MODE, &pmode,
                                                                  sizeof(pmode)) == HIPBLAS_STATUS_SUCCESS) &&
              (epi != EPI_VEC_BIAS || hipblasLtMatmulDescSetAttribute(p.op, HIPBLASLT_MATMUL_DESC_BIAS_DATA_TYPE,
                                                                      &btype, sizeof(btype)) ==
                                          HIPBLAS_STATUS_SUCCESS) &&
              hipblasLtMatrixLayoutCreate(&p.la, HIP_R_16F, k, m, k) == HIPBLAS_STATUS_SUCCESS &&
              hipblasLtMatrixLayoutCreate(&p.lb, HIP_R_16F, k, n, k) == HIPBLAS_STATUS_SUCCESS &&
              hipblasLtMatrixLayoutCreate(&p.lc, HIP_R_16F, m, n, m) == HIPBLAS_STATUS_SUCCESS &&
              hipblasLtMatmulPreferenceCreate(&pref) == HIPBLAS_STATUS_SUCCESS &&
              hipblasLtMatmulPreferenceSetAttribute(pref, HIPBLASLT_MATMUL_PREF_MAX_WORKSPACE_BYTES, &no_ws,
                                                    sizeof(no_ws)) == HIPBLAS_STATUS_SUCCESS &&
              hipblasLtMatmulAlgoGetHeuristic(g_handle[dev], p.op, p.la, p.lb, p.lc, p.lc, pref, 1, res, &nres) ==
                  HIPBLAS_STATUS_SUCCESS &&
              nres >= 1 && res[0].workspaceSize == 0;
    if (pref)
        hipblasLtMatmulPreferenceDestroy(pref);
    if (!ok) {
        if (p.op)
            hipblasLtMatmulDescDestroy(p.op);
        if (p.la)
            hipblasLtMatrixLayoutDestroy(p.la);
        if (p.lb)
            hipblasLtMatrixLayoutDestroy(p.lb);
        if (p.lc)
            hipblasLtMatrixLayoutDestroy(p.lc);
        p.op = nullptr;
        p.la = p.lb = p.lc = nullptr;
        g_plans[g_nplans++] = p;  // remembered as missing
        return hipErrorNotSupported;
    }
    p.valid = true;
    p.algo = res[0].algo;
    g_plans[g_nplans] = p;
    *out = &g_plans[g_nplans++];
    return hipSuccess;
}

// With epi != EPI_NONE: d = act(svec (a b) + beta c + bias) per row of D,
// svec and bias fp32 device vectors of m entries (bias only for
// EPI_VEC_BIAS), c (D's layout) only when beta != 0.
hipError_t gemm_nt(const void *a, const void *b, void *d, int m, int n, int k, hipStream_t st, int epi = EPI_NONE,
                   int act = 0, const float *svec = nullptr, const float *bias = nullptr, const void *c = nullptr,
                   float beta = 0.0f) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return e;
    if (dev < 0 || dev >= MAX_DEV)
        return hipErrorNotSupported;
    std::lock_guard<std::mutex> lk(g_mu);
    const Plan *p = nullptr;
    e = plan_for(dev, m, n, k, &p, true, epi, act);
    if (e != hipSuccess)
        return e;
    if (epi == EPI_VEC_BIAS &&
        hipblasLtMatmulDescSetAttribute(p->op, HIPBLASLT_MATMUL_DESC_BIAS_POINTER, &bias, sizeof(bias)) !=
            HIPBLAS_STATUS_SUCCESS)
        return hipErrorLaunchFailure;
    const float one = 1.0f;
    const void *alpha = epi == EPI_NONE ? (const void *)&one : (const void *)svec;
    return hipblasLtMatmul(g_handle[dev], p->op, alpha, a, p->la, b, p->lb, &beta, beta != 0.0f ? c : d, p->lc, d,
                           p->lc, &p->algo, nullptr, 0, st) == HIPBLAS_STATUS_SUCCESS
               ? hipSuccess
               : hipErrorLaunchFailure;
}

__device__ __forceinline__ float act_of(float u, int act) {
    if (act == ACT_GELU)
        return gelu_f32(u);
    if (act == ACT_RELU)
        return fmaxf(u, 0.0f);
    return u;
}

// eight scales and biases of channels c .. c + 7 (c % 8 == 0) as 16-byte loads
__device__ __forceinline__ void vec8(const float *s, const float *b, uint32_t c, float (&sc)[8], float (&bi)[8]) {
    const float4v s01 = s ? *reinterpret_cast<const float4v *>(s + c) : float4v{1.f, 1.f, 1.f, 1.f};
    const float4v s23 = s ? *reinterpret_cast<const float4v *>(s + c + 4) : float4v{1.f, 1.f, 1.f, 1.f};
    const float4v b01 = b ? *reinterpret_cast<const float4v *>(b + c) : float4v{0.f, 0.f, 0.f, 0.f};
    const float4v b23 = b ? *reinterpret_cast<const float4v *>(b + c + 4) : float4v{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int e = 0; e < 4; e++) {
        sc[e] = s01[e];
        sc[e + 4] = s23[e];
        bi[e] = b01[e];
        bi[e + 4] = b23[e];
    }
}

// The elementwise passes walk [rows][ch8] groups of eight channels with a
// grid stride that is a multiple of ch8 (grid_for), so a thread keeps one
// channel group -- its scales and biases in registers -- for every row it
// visits.  n8 < 2^31.

// h = act(s1 h + b1)
__global__ __launch_bounds__(256) void hidden_kernel(uint16_t *h, const float *s1, const float *b1, uint32_t n8,
                                                     uint32_t ec8, int act) {
    const uint32_t i0 = blockIdx.x * 256u + threadIdx.x, stride = gridDim.x * 256u;
    float sc[8], bi[8];
    vec8(s1, b1, (i0 % ec8) * 8, sc, bi);
    // two groups per step (both loads in flight before either store)
    for (uint32_t i = i0; i < n8; i += 2 * stride) {
        const bool two = i + stride < n8;
        u32x4 v[2];
        v[0] = *reinterpret_cast<const u32x4 *>(h + (size_t)i * 8);
        v[1] = *reinterpret_cast<const u32x4 *>(h + (size_t)(two ? i + stride : i) * 8);
#pragma unroll
        for (int j = 0; j < 2; j++)
#pragma unroll
            for (int e = 0; e < 4; e++) {
                const float u0 = fmaf(F16::lo(v[j][e]), sc[2 * e], bi[2 * e]);
                const float u1 = fmaf(F16::hi(v[j][e]), sc[2 * e + 1], bi[2 * e + 1]);
                if (act == ACT_GELU) {
                    // the fused kernels' packed GELU of u / 4, times 4
                    const half2v g = gelu_pk_f16_quarter(half2v{(_Float16)(0.25f * u0), (_Float16)(0.25f * u1)});
                    v[j][e] = __builtin_bit_cast(uint32_t, g * splat2(4.0f));
                } else {
                    v[j][e] = F16::pack2(act_of(u0, act), act_of(u1, act));
                }
            }
        *reinterpret_cast<u32x4 *>(h + (size_t)i * 8) = v[0];
        if (two)
            *reinterpret_cast<u32x4 *>(h + (size_t)(i + stride) * 8) = v[1];
    }
}

// y = s2 t + b2 + x
__global__ __launch_bounds__(256) void project_kernel(const uint16_t *t, const uint16_t *x, uint16_t *y,
                                                      const float *s2, const float *b2, uint32_t n8, uint32_t c8) {
    const uint32_t i0 = blockIdx.x * 256u + threadIdx.x, stride = gridDim.x * 256u;
    float sc[8], bi[8];
    vec8(s2, b2, (i0 % c8) * 8, sc, bi);
    for (uint32_t i = i0; i < n8; i += stride) {
        const u32x4 tv = *reinterpret_cast<const u32x4 *>(t + (size_t)i * 8);
        const u32x4 xv = *reinterpret_cast<const u32x4 *>(x + (size_t)i * 8);
        u32x4 out;
#pragma unroll
        for (int e = 0; e < 4; e++)
            out[e] = F16::pack2(fmaf(F16::lo(tv[e]), sc[2 * e], bi[2 * e]) + F16::lo(xv[e]),
                                fmaf(F16::hi(tv[e]), sc[2 * e + 1], bi[2 * e + 1]) + F16::hi(xv[e]));
        *reinterpret_cast<u32x4 *>(y + (size_t)i * 8) = out;
    }
}

// Depth-wise 3 x 3 conv of small images: a workgroup takes one image and 64
// channels, stages the zero-padded (H + 2) x (W + 2) slice in LDS (128 bytes
// a pixel, every input byte read once), and each thread keeps one group of
// 8 channels -- its 9 tap vectors, s0 and b0 in registers -- for every
// 32nd output pixel.  fp32 sums, s0, b0, rounded as the depth-wise kernel of
// the layer-by-layer block does.
constexpr int DW_LDS_MAX = 48 * 1024;

__global__ __launch_bounds__(256) void dw3_image_kernel(const uint16_t *x, uint16_t *d, const uint16_t *taps,
                                                        const float *s0, const float *b0, int H, int W, int C) {
    extern __shared__ __attribute__((aligned(16))) uint8_t sm[];
    const int slices = C / 64, n = blockIdx.x / slices, cs = blockIdx.x - n * slices;
    const int WP = W + 2, NPX = (H + 2) * WP;
    const uint16_t *xn = x + (size_t)n * H * W * C + cs * 64;
    for (int t = threadIdx.x; t < NPX * 8; t += 256) {
        const int px = t >> 3, pc = t & 7, r = px / WP - 1, c = px - (r + 1) * WP - 1;
        u32x4 v = {0u, 0u, 0u, 0u};
        if (r >= 0 && r < H && c >= 0 && c < W)
            v = *reinterpret_cast<const u32x4 *>(xn + ((size_t)r * W + c) * C + pc * 8);
        *reinterpret_cast<u32x4 *>(sm + px * 128 + pc * 16) = v;
    }
    const int g = threadIdx.x & 7, ch = cs * 64 + g * 8;
    u32x4 tp[9];
#pragma unroll
    for (int i = 0; i < 9; i++)
        tp[i] = *reinterpret_cast<const u32x4 *>(taps + (size_t)i * C + ch);
    float sc[8], bi[8];
    vec8(s0, b0, (uint32_t)ch, sc, bi);
    __syncthreads();
    for (int p = threadIdx.x >> 3; p < H * W; p += 32) {
        const int oh = p / W, ow = p - oh * W;
        float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int di = 0; di < 3; di++)
#pragma unroll
            for (int dj = 0; dj < 3; dj++) {
                const u32x4 v = *reinterpret_cast<const u32x4 *>(sm + ((oh + di) * WP + ow + dj) * 128 + g * 16);
                const u32x4 w = tp[di * 3 + dj];
#pragma unroll
                for (int q = 0; q < 4; q++) {
                    acc[2 * q] = fmaf(F16::lo(v[q]), F16::lo(w[q]), acc[2 * q]);
                    acc[2 * q + 1] = fmaf(F16::hi(v[q]), F16::hi(w[q]), acc[2 * q + 1]);
                }
            }
        u32x4 out;
#pragma unroll
        for (int q = 0; q < 4; q++)
            out[q] = F16::pack2(fmaf(acc[2 * q], sc[2 * q], bi[2 * q]), fmaf(acc[2 * q + 1], sc[2 * q + 1], bi[2 * q + 1]));
        *reinterpret_cast<u32x4 *>(d + (((size_t)n * H + oh) * W + ow) * C + ch) = out;
    }
}

hipError_t depthwise(const void *x, void *d, const BlockW &w, const Shape &s, hipStream_t st) {
    const size_t lds = (size_t)(s.H + 2) * (s.W + 2) * 128;
    if (s.k != 3 || s.C % 64 || lds > DW_LDS_MAX)
        return launch_depthwise(x, d, w, s, st);
    hipLaunchKernelGGL(dw3_image_kernel, dim3((unsigned)(s.N * (s.C / 64))), dim3(256), lds, st, (const uint16_t *)x,
                       (uint16_t *)d, (const uint16_t *)w.dw_w, w.s0, w.b0, s.H, s.W, s.C);
    return hipGetLastError();
}

// workgroups: enough for the groups (at most 8 per compute unit), a multiple
// of ch8 / gcd(ch8, 256) so that the stride keeps each thread's channels
unsigned grid_for(uint32_t n8, uint32_t ch8) {
    uint32_t g = ch8, b = 256;
    while (b) {
        const uint32_t r = g % b;
        g = b;
        b = r;
    }
    const uint32_t unit = ch8 / g;
    uint32_t nb = (n8 + 255) / 256, cap = (uint32_t)device_cu_count() * 8;
    if (nb > cap)
        nb = cap;
    nb = (nb + unit - 1) / unit * unit;
    return nb;
}

}  // namespace lgm

bool libgemm_ready(const Shape &s, hipStream_t st) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= lgm::MAX_DEV)
        return false;
    // inside a stream capture only plans made before are used: creating the
    // library handle allocates device memory, which a capture forbids
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(st, &cap) != hipSuccess)
        return false;
    const bool create = cap == hipStreamCaptureStatusNone;
    const int P = (int)((int64_t)s.N * s.H * s.W), C = s.C, EC = s.E * s.C;
    std::lock_guard<std::mutex> lk(lgm::g_mu);
    const lgm::Plan *p1 = nullptr, *p2 = nullptr, *p3 = nullptr;
    const bool ok = lgm::plan_for(dev, EC, P, C, &p1, create) == hipSuccess &&
                    lgm::plan_for(dev, C, P, EC, &p2, create) == hipSuccess;
    // the expand with s1, b1 and the activation in its epilogue, the project
    // with s2, b2 and the residual, when the library has algorithms for them
    // (else the separate passes run)
    if (ok) {
        lgm::plan_for(dev, EC, P, C, &p3, create, lgm::EPI_VEC_BIAS, s.act);
        lgm::plan_for(dev, C, P, EC, &p3, create, lgm::EPI_VEC_BIAS, ACT_NONE);
    }
    return ok;
}

// whether an epilogue plan exists (made by libgemm_ready): the expand's
// (project = false) or the project's
static bool fused_epilogue_ready(const Shape &s, bool project) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= lgm::MAX_DEV)
        return false;
    const int P = (int)((int64_t)s.N * s.H * s.W), C = s.C, EC = s.E * s.C;
    std::lock_guard<std::mutex> lk(lgm::g_mu);
    const lgm::Plan *p = nullptr;
    return project ? lgm::plan_for(dev, C, P, EC, &p, false, lgm::EPI_VEC_BIAS, ACT_NONE) == hipSuccess
                   : lgm::plan_for(dev, EC, P, C, &p, false, lgm::EPI_VEC_BIAS, s.act) == hipSuccess;
}

bool libgemm_applies(const Shape &s) {
    const int64_t P = (int64_t)s.N * s.H * s.W;
    return !s.bf16 && s.C == 512 && s.E * s.C <= 4096 && P >= 4096 && P < ((int64_t)1 << 30) / (s.E * s.C);
}

size_t libgemm_scratch_bytes(const Shape &s) {
    const size_t P = (size_t)s.N * s.H * s.W;
    const size_t d = (P * s.C * 2 + 255) & ~(size_t)255, h = (P * s.E * s.C * 2 + 255) & ~(size_t)255;
    return 2 * d + h;
}

hipError_t launch_block_libgemm(const void *x, void *y, const BlockW &w, const Shape &s, void *scratch,
                                hipStream_t st) {
    if (!libgemm_applies(s))
        return hipErrorNotSupported;
    const int64_t P = (int64_t)s.N * s.H * s.W;
    const int C = s.C, EC = s.E * s.C;
    const size_t dbytes = ((size_t)P * C * 2 + 255) & ~(size_t)255;
    const size_t hbytes = ((size_t)P * EC * 2 + 255) & ~(size_t)255;
    uint16_t *d = (uint16_t *)scratch;
    uint16_t *h = (uint16_t *)((char *)scratch + dbytes);
    uint16_t *t = (uint16_t *)((char *)scratch + dbytes + hbytes);
    hipError_t e = lgm::depthwise(x, d, w, s, st);
    if (e != hipSuccess)
        return e;
    if (w.s1 && w.b1 && fused_epilogue_ready(s, false)) {
        // s1, b1 and the activation in the expand's epilogue
        e = lgm::gemm_nt(w.w1, d, h, EC, (int)P, C, st, lgm::EPI_VEC_BIAS, s.act, w.s1, w.b1);
        if (e != hipSuccess)
            return e;
    } else {
        e = lgm::gemm_nt(w.w1, d, h, EC, (int)P, C, st);
        if (e != hipSuccess)
            return e;
        const uint32_t nh = (uint32_t)(P * EC / 8);
        hipLaunchKernelGGL(lgm::hidden_kernel, dim3(lgm::grid_for(nh, EC / 8)), dim3(256), 0, st, h, w.s1, w.b1,
                           nh, (uint32_t)(EC / 8), s.act);
        e = hipGetLastError();
        if (e != hipSuccess)
            return e;
    }
    if (w.s2 && w.b2 && fused_epilogue_ready(s, true))  // y = s2 (W2 h) + x + b2 in the epilogue
        return lgm::gemm_nt(w.w2, h, y, C, (int)P, EC, st, lgm::EPI_VEC_BIAS, ACT_NONE, w.s2, w.b2, x, 1.0f);
    e = lgm::gemm_nt(w.w2, h, t, C, (int)P, EC, st);
    if (e != hipSuccess)
        return e;
    const uint32_t ny = (uint32_t)(P * C / 8);
    hipLaunchKernelGGL(lgm::project_kernel, dim3(lgm::grid_for(ny, C / 8)), dim3(256), 0, st, t,
                       (const uint16_t *)x, (uint16_t *)y, w.s2, w.b2, ny, (uint32_t)(C / 8));
    return hipGetLastError();
}

}  // namespace cf
