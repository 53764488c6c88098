// cf_mbconv.hip -- block fusion of the paper's MBConv block with Squeeze &
// Excitation (Sec. 5.4 of Lavin, arXiv:2404.03617; the kernel of Sec. 5.4.1,
// Fig. f:mbconv-block-fusion-tensor-machine):
//   U = SiLU(s1 (X W1^T) + b1)                     expand to E*C hidden channels
//   V = SiLU(s2 gconv3x3(U) + b2)                  grouped conv, group width 8
//   g = sigmoid(We ReLU(Wr mean_hw(V) + br) + be)  squeeze & excitation
//   Y = X + s3 (W2 diag(g) V) + b3                 project, residual
//
// As in the paper, a work item is one image and one group of 64 hidden
// channels, and the expand and conv layers of that group run on one
// processor without other work items:
//  1. expand: the group's 64 rows of W1 against every pixel of the image
//     (v_mfma_f32_16x16x32, x read straight from global memory as B
//     fragments, one K step prefetched), SiLU in fp32, rounded into an LDS
//     buffer with a zero border;
//  2. grouped conv of the 64 channels (8 groups of 8, self-contained) as one
//     product per tap column: 16 columns x 2 output rows against K = 4 halo
//     rows x 8 channels; SiLU; V goes to the image's exchange buffer in
//     global memory, and its channel sums are reduced in registers (lane
//     shuffles in a fixed order);
//  3. the group's share of the squeeze product, Wr[:, group] . mean(V), to a
//     workspace slot;
//  4. the per-image barrier: every work item of the image has written its V
//     and its squeeze share;
//  5. the squeeze (shares added in group order), ReLU, and the excitation
//     and sigmoid for all E*C hidden channels;
//  6. the projection: the image's output is cut into tiles of 16 pixels x 16
//     channels, dealt round-robin to the image's work items; each tile is a
//     product over all E*C hidden channels of W2 (gate folded into its
//     fragments) and the exchanged V, then s3, b3 and the residual, and y is
//     written once.
// Where the paper adds the groups' projections into y with atomics, the
// work items here exchange the (4x smaller) gated-layer input instead; the
// result is deterministic and needs one synchronisation per image.  The
// barrier follows every read of x for the image, so y may be x itself.
//
// Coherence: the exchanged data (V, squeeze shares, counters) moves only
// through device-scope atomic loads and stores, which the memory system keeps
// coherent across the XCDs' L2 caches without write-backs or invalidations.
// A wave waits for its outstanding stores (vmcnt 0) before its workgroup
// signals arrival, the ordering the compiler itself uses for device-scope
// release; full release/acquire fences would write back and invalidate the
// whole L2 at every barrier, which costs more than the rest of the kernel.
//
// The barrier needs every work item of an image resident at once: the grid is
// launched cooperatively with at most as many workgroups as fit on the
// device, `slots` images in flight, each slot's workgroups walking the same
// sequence of images; the exchange buffer of a slot alternates between two
// halves, so an image's V never overwrites the previous image's while it is
// read.  The wait is bounded; one that gives up sets a flag in the workspace,
// the later waits of the launch are skipped, and the kernel always ends.
//
// Images up to 16 x 16 (the late-stage shapes the paper targets); C a
// multiple of 16; E*C a multiple of 64 and at most 4096; 1 <= R <= 256.
#include "cf_device.h"
#include "cf_kernels.h"

namespace cf {
namespace mbc {

constexpr int GH = 64;            // hidden channels per work item
constexpr int HMAX = 16, WMAX = 16;
constexpr int UC = WMAX + 2;      // columns of the U buffer (zero border)
constexpr int PB = 2 * GH + 16;   // LDS bytes per pixel: an odd multiple of 16, conflict-free 16-B reads
constexpr int RMAX = 256;
constexpr int ECMAX = 4096;
constexpr int SPIN_LIMIT = 1 << 20;

struct Args {
    const uint16_t *x;
    uint16_t *y;
    const uint16_t *w1;            // [EC][C]
    const float *s1, *b1;
    const uint16_t *gw;            // [3][3][EC][8]
    const float *s2, *b2;
    const uint16_t *wr;            // [R][EC]
    const float *br;
    const uint16_t *we;            // [EC][R]
    const float *be;
    const uint16_t *w2;            // [C][EC]
    const float *s3, *b3;
    int *flag;                     // nonzero once a barrier wait gave up
    int *cnt;                      // [N] arrivals per image
    float *sq;                     // [N][G][R] squeeze shares
    uint16_t *vx;                  // [2][slots][P][EC] exchanged conv output
    int N, H, W, C, EC, R, G;
    int slots;
    int xcd_map;                   // 1: the workgroups of a slot share an XCD
    uint32_t off_gate, off_z, off_cs;  // LDS layout (U at 0)
};

__device__ __forceinline__ u32x4 ld16(const void *p) { return *reinterpret_cast<const u32x4 *>(p); }

// device-scope atomic 64-bit store / load (the exchange of V)
__device__ __forceinline__ void st8_dev(uint16_t *p, u32x2 v) {
    __hip_atomic_store(reinterpret_cast<unsigned long long *>(p), __builtin_bit_cast(unsigned long long, v),
                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ u32x2 ld8_dev(const uint16_t *p) {
    return __builtin_bit_cast(u32x2, __hip_atomic_load(reinterpret_cast<const unsigned long long *>(p),
                                                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
}

__device__ __forceinline__ float silu_f32(float u) { return u * __builtin_amdgcn_rcpf(1.0f + __expf(-u)); }
__device__ __forceinline__ float sigmoid_f32(float u) { return __builtin_amdgcn_rcpf(1.0f + __expf(-u)); }

// Every thread's device-scope stores so far are complete when the workgroup
// adds its arrival to cnt; returns once cnt reaches target (or a wait gave up).
__device__ __forceinline__ void image_barrier(int *cnt, int target, int *flag) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (threadIdx.x == 0) {
        __hip_atomic_fetch_add(cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (__hip_atomic_load(flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0) {
            int spins = 0;
            while (__hip_atomic_load(cnt, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
                if (++spins > SPIN_LIMIT) {
                    __hip_atomic_store(flag, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    break;
                }
                // another workgroup gave up: stop waiting too
                if ((spins & 63) == 0 && __hip_atomic_load(flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))
                    break;
                __builtin_amdgcn_s_sleep(1);
            }
        }
    }
    __syncthreads();
}

template <typename T, int NWV, int NPW>
struct MB {
    static constexpr int NT = NWV * 64;

    static __device__ void run(const Args &a, uint8_t *smem) {
        const int tid = threadIdx.x, lane = tid & 63;
        const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
        const int q = lane >> 4, jl = lane & 15;
        const int M = gridDim.x;
        int lin = blockIdx.x;
        if (a.xcd_map)  // workgroup i runs on XCD i % 8
            lin = (int)(blockIdx.x % 8) * (M / 8) + (int)(blockIdx.x / 8);
        const int g = lin % a.G, slot = lin / a.G;
        const int C = a.C, EC = a.EC, R = a.R, G = a.G;
        const int P = a.H * a.W;
        const int RP = (a.H + 1) / 2;
        const int h0 = g * GH;  // first hidden channel of the group
        uint8_t *U = smem;
        float *gate = reinterpret_cast<float *>(smem + a.off_gate);  // [EC]
        float *zl = reinterpret_cast<float *>(smem + a.off_z);       // [R]
        float *csum = reinterpret_cast<float *>(smem + a.off_cs);    // [64]

        // the U border (row 0, rows past H, column 0, columns past W) stays zero
        for (uint32_t i = tid; i < a.off_gate / 16; i += NT)
            reinterpret_cast<u32x4 *>(smem)[i] = u32x4{0u, 0u, 0u, 0u};
        __syncthreads();

        int it = 0;
        for (int n = slot; n < a.N; n += a.slots, it++) {
            const uint16_t *xn = a.x + (size_t)n * P * C;
            uint16_t *vx = a.vx + ((size_t)(it & 1) * a.slots + slot) * P * EC;

            // ---- 1. expand + SiLU into U; wave wv takes the 16-pixel tiles wv + NWV i
            {
                float4v acc[4][NPW];
#pragma unroll
                for (int mt = 0; mt < 4; mt++)
#pragma unroll
                    for (int i = 0; i < NPW; i++)
                        acc[mt][i] = float4v{0.f, 0.f, 0.f, 0.f};
                const int ks = (C + 31) / 32;
                auto load = [&](int kk, u32x4 *av, u32x4 *bv) {
                    const int k0 = 32 * kk + 8 * q;
                    const bool kin = k0 < C;  // C % 32 == 16: the last step is half padding
#pragma unroll
                    for (int mt = 0; mt < 4; mt++)
                        av[mt] = kin ? ld16(a.w1 + (size_t)(h0 + 16 * mt + jl) * C + k0) : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
                    for (int i = 0; i < NPW; i++) {
                        const int p = 16 * (wv + NWV * i) + jl;
                        bv[i] = kin && p < P ? ld16(xn + (size_t)p * C + k0) : u32x4{0u, 0u, 0u, 0u};
                    }
                };
                auto mma = [&](const u32x4 *av, const u32x4 *bv) {
#pragma unroll
                    for (int mt = 0; mt < 4; mt++)
#pragma unroll
                        for (int i = 0; i < NPW; i++)
                            acc[mt][i] = T::mfma(av[mt], bv[i], acc[mt][i]);
                };
                u32x4 a0[4], b0[NPW], a1[4], b1[NPW];
                load(0, a0, b0);
                for (int kk = 0; kk < ks; kk += 2) {
                    if (kk + 1 < ks)
                        load(kk + 1, a1, b1);
                    mma(a0, b0);
                    if (kk + 1 < ks) {
                        if (kk + 2 < ks)
                            load(kk + 2, a0, b0);
                        mma(a1, b1);
                    }
                }
#pragma unroll
                for (int mt = 0; mt < 4; mt++) {
                    const int hl = 16 * mt + 4 * q;  // local hidden channels hl .. hl+3 of this lane
                    float sc[4], bi[4];
#pragma unroll
                    for (int e = 0; e < 4; e++) {
                        sc[e] = a.s1 ? a.s1[h0 + hl + e] : 1.0f;
                        bi[e] = a.b1 ? a.b1[h0 + hl + e] : 0.0f;
                    }
#pragma unroll
                    for (int i = 0; i < NPW; i++) {
                        const int p = 16 * (wv + NWV * i) + jl;
                        if (p >= P)
                            continue;
                        float u[4];
#pragma unroll
                        for (int e = 0; e < 4; e++)
                            u[e] = silu_f32(fmaf(acc[mt][i][e], sc[e], bi[e]));
                        const int r = p / a.W, c = p - r * a.W;
                        *reinterpret_cast<u32x2 *>(U + (uint32_t)((r + 1) * UC + c + 1) * PB + (uint32_t)hl * 2) =
                            u32x2{T::pack2(u[0], u[1]), T::pack2(u[2], u[3])};
                    }
                }
            }
            __syncthreads();

            // ---- 2. grouped conv + SiLU -> exchange buffer, channel sums.  A rows
            //      (s, o): output row 2rp+s, channel o of the 8-group; K (t, j):
            //      halo row 2rp+t, input channel j
            {
                const int cs = jl >> 3, co = jl & 7;
                const int ti = q - cs;  // the tap row this lane's K slice meets
                const bool tap_ok = ti >= 0 && ti <= 2;
                for (int gg = wv; gg < 8; gg += NWV) {
                    u32x4 av[3];
#pragma unroll
                    for (int dj = 0; dj < 3; dj++)
                        av[dj] = tap_ok ? ld16(a.gw + ((size_t)(ti * 3 + dj) * EC + h0 + 8 * gg + co) * 8)
                                        : u32x4{0u, 0u, 0u, 0u};
                    const int hl = 8 * gg + 4 * (q & 1);  // output channels of this lane's D rows
                    float sc[4], bi[4], sum[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int e = 0; e < 4; e++) {
                        sc[e] = a.s2 ? a.s2[h0 + hl + e] : 1.0f;
                        bi[e] = a.b2 ? a.b2[h0 + hl + e] : 0.0f;
                    }
                    for (int rp = 0; rp < RP; rp++) {
                        float4v acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                        for (int dj = 0; dj < 3; dj++) {
                            const u32x4 bv = *reinterpret_cast<const u32x4 *>(
                                U + (uint32_t)((2 * rp + q) * UC + jl + dj) * PB + (uint32_t)gg * 16);
                            acc = T::mfma(av[dj], bv, acc);
                        }
                        const int r = 2 * rp + (q >> 1), c = jl;
                        if (r < a.H && c < a.W) {
                            float u[4];
#pragma unroll
                            for (int e = 0; e < 4; e++) {
                                u[e] = silu_f32(fmaf(acc[e], sc[e], bi[e]));
                                sum[e] += u[e];
                            }
                            st8_dev(vx + (size_t)(r * a.W + c) * EC + h0 + hl,
                                    u32x2{T::pack2(u[0], u[1]), T::pack2(u[2], u[3])});
                        }
                    }
                    // sum over the 16 columns (lane bits 0-3) and the two rows of a
                    // pair (lane bit 5); lanes 0 and 16 hold channels hl .. hl+3
#pragma unroll
                    for (int e = 0; e < 4; e++) {
#pragma unroll
                        for (int m = 1; m <= 8; m <<= 1)
                            sum[e] += __shfl_xor(sum[e], m);
                        sum[e] += __shfl_xor(sum[e], 32);
                    }
                    if (jl == 0 && q < 2) {
#pragma unroll
                        for (int e = 0; e < 4; e++)
                            csum[hl + e] = sum[e];
                    }
                }
            }
            __syncthreads();

            // ---- 3. the group's share of the squeeze: Wr[:, group] . mean(V)
            if (tid < R) {
                const float inv = 1.0f / (float)P;
                float s = 0.0f;
                const uint16_t *wrow = a.wr + (size_t)tid * EC + h0;
#pragma unroll
                for (int c = 0; c < GH; c += 8) {
                    Pack8 w;
                    w.u = ld16(wrow + c);
#pragma unroll
                    for (int e = 0; e < 4; e++)
                        s += T::lo(w.w[e]) * csum[c + 2 * e] + T::hi(w.w[e]) * csum[c + 2 * e + 1];
                }
                __hip_atomic_store(a.sq + ((size_t)n * G + g) * R + tid, s * inv, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
            }

            // ---- 4. every work item of image n has written its V and its share
            image_barrier(a.cnt + n, G, a.flag);

            // ---- 5. squeeze (shares in group order), excitation, gates of all channels
            for (int r = tid; r < R; r += NT) {
                float s = a.br ? a.br[r] : 0.0f;
                for (int gg = 0; gg < G; gg++)
                    s += __hip_atomic_load(a.sq + ((size_t)n * G + gg) * R + r, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT);
                zl[r] = s > 0.0f ? s : 0.0f;
            }
            __syncthreads();
            for (int c = tid; c < EC; c += NT) {
                const uint16_t *wrow = a.we + (size_t)c * R;
                float s = a.be ? a.be[c] : 0.0f;
                int r = 0;
                if ((R & 7) == 0) {
                    for (; r < R; r += 8) {
                        Pack8 w;
                        w.u = ld16(wrow + r);
#pragma unroll
                        for (int e = 0; e < 4; e++)
                            s += T::lo(w.w[e]) * zl[r + 2 * e] + T::hi(w.w[e]) * zl[r + 2 * e + 1];
                    }
                }
                for (; r < R; r++)
                    s += T::lo((uint32_t)wrow[r]) * zl[r];
                gate[c] = sigmoid_f32(s);
            }
            __syncthreads();

            // ---- 6. output tiles t = g + G (wv + NWV i): 16 pixels x 16 channels, K = EC
            {
                const int PT = (P + 15) / 16, T16 = PT * (C / 16);
                const int kst = EC / 32;
                for (int t = g + G * wv; t < T16; t += G * NWV) {
                    const int pt = t % PT, ot = t / PT;
                    const int p = 16 * pt + jl;
                    const bool pin = p < P;
                    const uint16_t *wrow = a.w2 + (size_t)(16 * ot + jl) * EC + 8 * q;
                    const uint16_t *vrow = vx + (size_t)(pin ? p : 0) * EC + 8 * q;
                    float4v acc = {0.f, 0.f, 0.f, 0.f};
                    auto load = [&](int kk, u32x4 &w, u32x4 &v) {
                        w = ld16(wrow + 32 * kk);
                        if (pin) {
                            const u32x2 lo = ld8_dev(vrow + 32 * kk), hi = ld8_dev(vrow + 32 * kk + 4);
                            v = u32x4{lo[0], lo[1], hi[0], hi[1]};
                        } else {
                            v = u32x4{0u, 0u, 0u, 0u};
                        }
                    };
                    auto mma = [&](int kk, const u32x4 &w, const u32x4 &v) {
                        const float4v g0 = *reinterpret_cast<const float4v *>(gate + 32 * kk + 8 * q);
                        const float4v g1 = *reinterpret_cast<const float4v *>(gate + 32 * kk + 8 * q + 4);
                        u32x4 av;
                        av[0] = T::pack2(T::lo(w[0]) * g0[0], T::hi(w[0]) * g0[1]);
                        av[1] = T::pack2(T::lo(w[1]) * g0[2], T::hi(w[1]) * g0[3]);
                        av[2] = T::pack2(T::lo(w[2]) * g1[0], T::hi(w[2]) * g1[1]);
                        av[3] = T::pack2(T::lo(w[3]) * g1[2], T::hi(w[3]) * g1[3]);
                        acc = T::mfma(av, v, acc);
                    };
                    u32x4 w0, v0, w1, v1;
                    load(0, w0, v0);
                    for (int kk = 0; kk < kst; kk += 2) {
                        load(kk + 1, w1, v1);  // kst is even: EC is a multiple of 64
                        mma(kk, w0, v0);
                        if (kk + 2 < kst)
                            load(kk + 2, w0, v0);
                        mma(kk + 1, w1, v1);
                    }
                    if (pin) {
                        const int o = 16 * ot + 4 * q;
                        const float4v sc =
                            a.s3 ? *reinterpret_cast<const float4v *>(a.s3 + o) : float4v{1.f, 1.f, 1.f, 1.f};
                        const float4v bi =
                            a.b3 ? *reinterpret_cast<const float4v *>(a.b3 + o) : float4v{0.f, 0.f, 0.f, 0.f};
                        const size_t e = ((size_t)n * P + p) * C + o;
                        const u32x2 xv = *reinterpret_cast<const u32x2 *>(a.x + e);
                        u32x2 out;
                        out[0] = T::pack2(T::lo(xv[0]) + fmaf(acc[0], sc[0], bi[0]),
                                          T::hi(xv[0]) + fmaf(acc[1], sc[1], bi[1]));
                        out[1] = T::pack2(T::lo(xv[1]) + fmaf(acc[2], sc[2], bi[2]),
                                          T::hi(xv[1]) + fmaf(acc[3], sc[3], bi[3]));
                        *reinterpret_cast<u32x2 *>(a.y + e) = out;
                    }
                }
            }
            // U, the gates and the sums are rewritten only after the next
            // image's first __syncthreads, which every thread reaches after
            // its last read of them here
        }
    }
};

template <typename T, int NWV, int NPW>
__global__ __launch_bounds__(NWV * 64) void mbconv_kernel(Args a) {
    extern __shared__ __attribute__((aligned(256))) uint8_t smem[];
    MB<T, NWV, NPW>::run(a, smem);
}

// clears the give-up flag and the arrival counters (a kernel rather than a
// memset, so that a captured graph replays it faithfully)
__global__ void clear_kernel(int *p, int n) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n)
        p[i] = 0;
}

struct Layout {
    uint32_t off_gate, off_z, off_cs, lds;
    int nwv;
};

// LDS layout for an H x W image.  U holds the border row above the image,
// its H rows, and zero rows below up to an even count of row pairs plus one
// (the conv reads halo rows 2rp .. 2rp+3 for every row pair rp); then the
// gates of all EC channels, the squeeze vector and the group's channel sums.
Layout layout(int H, int W, int EC, int R) {
    Layout l;
    const int P = H * W;
    l.nwv = P > 128 ? 8 : 4;
    const uint32_t urows = (uint32_t)(2 * ((H + 1) / 2) + 2);
    l.off_gate = urows * UC * PB;
    l.off_z = l.off_gate + (uint32_t)EC * 4;
    l.off_cs = l.off_z + (((uint32_t)R * 4 + 15) & ~15u);
    l.lds = l.off_cs + GH * 4;
    return l;
}

size_t head_bytes(int N) { return 256 + (((size_t)N * 4 + 255) & ~(size_t)255); }
size_t sq_bytes(int N, int G, int R) { return ((size_t)N * G * R * 4 + 255) & ~(size_t)255; }

}  // namespace mbc

bool mbconv_supported(int H, int W, int C, int E, int R) {
    return H >= 1 && W >= 1 && H <= mbc::HMAX && W <= mbc::WMAX && C >= 16 && C % 16 == 0 && E >= 1 &&
           (E * C) % mbc::GH == 0 && E * C <= mbc::ECMAX && R >= 1 && R <= mbc::RMAX;
}

namespace {

// The kernel instance for the shape and its launch size.
const void *mbconv_kernel_for(int H, int W, int EC, int R, int bf16, mbc::Layout *l, int *nt) {
    *l = mbc::layout(H, W, EC, R);
    *nt = l->nwv * 64;
    const int P = H * W;
    if (l->nwv == 8)
        return bf16 ? (const void *)mbc::mbconv_kernel<BF16, 8, 2> : (const void *)mbc::mbconv_kernel<F16, 8, 2>;
    if (P > 64)
        return bf16 ? (const void *)mbc::mbconv_kernel<BF16, 4, 2> : (const void *)mbc::mbconv_kernel<F16, 4, 2>;
    return bf16 ? (const void *)mbc::mbconv_kernel<BF16, 4, 1> : (const void *)mbc::mbconv_kernel<F16, 4, 1>;
}

}  // namespace

hipError_t mbconv_resident_slots(int H, int W, int C, int E, int R, int bf16, int *slots) {
    mbc::Layout l;
    int nt = 0;
    const void *kf = mbconv_kernel_for(H, W, E * C, R, bf16, &l, &nt);
    hipError_t e = allow_full_lds(kf);
    if (e != hipSuccess)
        return e;
    int per_cu = 0;
    if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kf, nt, l.lds)) != hipSuccess)
        return e;
    *slots = per_cu * device_cu_count() / (E * C / mbc::GH);
    return hipSuccess;
}

size_t mbconv_workspace_bytes(int N, int H, int W, int C, int E, int R, int slots) {
    const int G = E * C / mbc::GH;
    return mbc::head_bytes(N) + mbc::sq_bytes(N, G, R) + 2 * (size_t)slots * H * W * E * C * 2;
}

hipError_t launch_mbconv(const void *x, void *y, const MBConvW &w, int N, int H, int W, int C, int E, int R,
                         int bf16, void *ws, size_t ws_bytes, hipStream_t st) {
    mbc::Args a{};
    a.x = (const uint16_t *)x;
    a.y = (uint16_t *)y;
    a.w1 = (const uint16_t *)w.w1;
    a.s1 = w.s1;
    a.b1 = w.b1;
    a.gw = (const uint16_t *)w.gw;
    a.s2 = w.s2;
    a.b2 = w.b2;
    a.wr = (const uint16_t *)w.wr;
    a.br = w.br;
    a.we = (const uint16_t *)w.we;
    a.be = w.be;
    a.w2 = (const uint16_t *)w.w2;
    a.s3 = w.s3;
    a.b3 = w.b3;
    a.N = N;
    a.H = H;
    a.W = W;
    a.C = C;
    a.EC = E * C;
    a.R = R;
    a.G = a.EC / mbc::GH;
    mbc::Layout l;
    int nt = 0;
    const void *kf = mbconv_kernel_for(H, W, a.EC, R, bf16, &l, &nt);
    a.off_gate = l.off_gate;
    a.off_z = l.off_z;
    a.off_cs = l.off_cs;
    const size_t fixed = mbc::head_bytes(N) + mbc::sq_bytes(N, a.G, R);
    const size_t per_slot = 2 * (size_t)H * W * a.EC * 2;
    if (ws_bytes < fixed + per_slot)
        return hipErrorInvalidValue;
    char *base = (char *)ws;
    a.flag = (int *)base;
    a.cnt = (int *)(base + 256);
    a.sq = (float *)(base + mbc::head_bytes(N));
    // every work item of an image must be resident with the others (the
    // barrier waits for them): the grid holds at most what fits on the device
    // and is launched cooperatively, which the runtime refuses rather than
    // run partly
    int slots = 0;
    hipError_t e = mbconv_resident_slots(H, W, C, E, R, bf16, &slots);
    if (e != hipSuccess)
        return e;
    if (slots < 1)
        return hipErrorInvalidConfiguration;  // the groups of one image do not fit at once
    if (slots > N)
        slots = N;
    if ((size_t)slots * per_slot > ws_bytes - fixed)
        slots = (int)((ws_bytes - fixed) / per_slot);
    a.slots = slots;
    a.vx = (uint16_t *)(base + fixed);
    const int grid = slots * a.G;
    // a slot's workgroups on one XCD when the grid allows it
    a.xcd_map = grid % 8 == 0 && (grid / 8) % a.G == 0 ? 1 : 0;
    hipLaunchKernelGGL(mbc::clear_kernel, dim3((64 + N + 255) / 256), dim3(256), 0, st, a.flag, 64 + N);
    if ((e = hipGetLastError()) != hipSuccess)
        return e;
    void *args[] = {&a};
    return hipLaunchCooperativeKernel(kf, dim3(grid), dim3(nt), args, l.lds, st);
}

}  // namespace cf
