// cf_slice.hip -- the fused block for a handful of pixels (N*H*W <= 64)
// without a workspace.  There the weights, not the activations, are the bytes
// (Sec. 4.1.2), and a kernel whose workgroups each own a tile of pixels has
// one or two workgroups of work.  Here workgroup j owns output channels
// 32j .. 32j + 31 of every pixel (the output-channel partition of the block's
// last layer, Sec. 5.3.1) and recomputes the expand in full; its 8 waves
// split the hidden chunks and add their projections in LDS in wave order, so
// no partial sum leaves the workgroup and no caller memory is needed.
//  1. x (every pixel) and the depth-wise taps are copied to LDS; the
//     depth-wise conv writes D = s0 * conv + b0 to LDS over the taps (fp32
//     accumulation; an item is a pixel and 8 channels, a thread keeps one
//     channel chunk and its items in registers);
//  2. wave w runs hidden chunks w, w + 8, ...: the expand on
//     v_mfma_f32_16x16x32 (W1 straight from global memory, four adjacent
//     lanes on 64 contiguous bytes of a row, four groups of K steps ahead,
//     each dword then moved to its fragment lane by ds_bpermute one group
//     ahead of its products; D fragments from LDS), phi(s1 u + b1) in fp32
//     (s1, b1 staged in LDS), one exchange of quads between lanes l and
//     l ^ 16, and the projection onto the workgroup's 32 output channels
//     (v_mfma_f32_32x32x16, W2 rows in the tau order of cf_fused_impl.h as
//     the A operand, loaded one chunk ahead);
//  3. the waves' projections are summed in wave order and
//     y = x + s2 * sum + b2 is stored.
#include <algorithm>

#include "cf_device.h"
#include "cf_fused_impl.h"
#include "cf_kernels.h"

namespace cf {
namespace slice {

using fused::float16v;
using fused::mfma32;
using fused::tau_row;

constexpr int NW = 8, NT = NW * 64;
constexpr int PMAX = 64;  // pixels of a launch: at most two 32-pixel blocks

struct Args {
    const uint16_t *x, *dw_w, *w1, *w2;
    const float *s0, *b0, *s1, *b1, *s2, *b2;
    uint16_t *y;
    int H, W, HW, EC, k, act, P;
    uint32_t off_zero, off_d;  // LDS: a zero 16-byte piece, the D pixels
};

// GELU(u) = u * Phi(u) with erf from Abramowitz & Stegun 7.1.26
// (|error| <= 1.5e-7): a reciprocal, an exponential and no branch, where the
// library erff takes two divergent paths of about 30 instructions.
__device__ __forceinline__ float gelu_as(float u) {
    const float x = fabsf(u) * 0.70710678118654752f;
    const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, x, 1.0f));
    float q = fmaf(1.061405429f, t, -1.453152027f);
    q = fmaf(q, t, 1.421413741f);
    q = fmaf(q, t, -0.284496736f);
    q = fmaf(q, t, 0.254829592f);
    q *= t;
    const float e = __builtin_amdgcn_exp2f(x * x * -1.4426950408889634f);  // exp(-x^2)
    const float erf_x = fmaf(-q, e, 1.0f);
    const float hu = 0.5f * u;
    return fmaf(hu, copysignf(erf_x, u), hu);
}

template <typename T, int C, int PB>
struct Kern {
    static constexpr int KS = C / 32, C8 = C / 8;      // 32-element K steps of the expand
    static constexpr int KG = KS >= 16 ? 2 : 1;         // K steps per W1 fragment group (4 KB or 2 KB a wave)
    static constexpr int NG = KS / KG;                  // groups per chunk (a multiple of the ring's 4)
    static constexpr uint32_t XP = C * 2;               // LDS bytes per x pixel
    static constexpr uint32_t DP = C * 2 + 16;          // LDS bytes per D pixel (16-byte pad)
    static constexpr int NPX = PB * 32;
    static constexpr int IT = NPX * C8 / NT;            // depth-wise items (and x pieces) per thread
    static_assert(NT % C8 == 0 && IT >= 1 && IT * NT == NPX * C8, "item split");
    static_assert(NG % 4 == 0, "whole passes of the four-group ring per chunk");

    static __device__ float act(float u, int a) {
        return a == ACT_GELU ? gelu_as(u) : a == ACT_RELU ? fmaxf(u, 0.0f) : u;
    }

    static __device__ void run(const Args &a, uint8_t *smem) {
        const int tid = threadIdx.x, lane = tid & 63;
        const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform: scalar loop control
        const int h = lane >> 5, m = lane & 31;
        const int o0 = blockIdx.x * 32;  // the workgroup's first output channel

        // 1a. every pixel of x into LDS (pixels past P: zero) and the zero piece
        {
            u32x4 v[IT];
#pragma unroll
            for (int u = 0; u < IT; u++) {
                const int i = u * NT + tid, px = i / C8, cq = i - px * C8;
                v[u] = px < a.P ? *reinterpret_cast<const u32x4 *>(a.x + (size_t)px * C + cq * 8)
                                : u32x4{0u, 0u, 0u, 0u};
            }
#pragma unroll
            for (int u = 0; u < IT; u++) {
                const int i = u * NT + tid, px = i / C8, cq = i - px * C8;
                *reinterpret_cast<u32x4 *>(smem + (uint32_t)px * XP + (uint32_t)cq * 16) = v[u];
            }
            if (tid == 0)
                *reinterpret_cast<u32x4 *>(smem + a.off_zero) = u32x4{0u, 0u, 0u, 0u};
            // the taps [k][k][C] into the D region (D is written after they are used)
            const int tp = a.k * a.k * C8;
            for (int i = tid; i < tp; i += NT)
                *reinterpret_cast<u32x4 *>(smem + a.off_d + (uint32_t)i * 16) =
                    *reinterpret_cast<const u32x4 *>(a.dw_w + (size_t)i * 8);
        }
        __syncthreads();

        // The wave's hidden chunks.  The expand runs on 16 x 16 x 32
        // products: A = W1 rows 32 ch + 16 mt + r (r = lane & 15), elements
        // 32 ks + 8 q .. + 7 (q = lane >> 4); B = D, pixel 32 pb + 16 nt + r, channels
        // 32 ks + 8 q ..  Lane (q, r) then holds hidden 32 ch + 16 mt + 4 q + i
        // of pixel 32 pb + 16 nt + r.  The projection (32 x 32 x 16, W2 rows
        // o0 + tau(m) as the A operand) takes hidden 16 kk .. 16 kk + 15 of
        // the chunk in natural order as its K step kk: lane (h, m) with
        // m = 16 b + r needs hidden 16 kk + 8 h .. + 7 of pixel m; it holds
        // the quad 16 kk + 8 h + 4 b of that pixel and receives the quad
        // 16 kk + 8 h + 4 (1 - b) from lane l ^ 16, to which it sends its
        // values of the partner's pixel.
        const int NCH = a.EC / 32;
        const int r = lane & 15, q = lane >> 4, b = q & 1;
        const uint32_t dbase = a.off_d + (uint32_t)r * DP + (uint32_t)q * 16;
        // W1 is read with lanes 4 i .. 4 i + 3 on 64 contiguous bytes of row i
        // (the memory unit merges adjacent lanes only: in the fragment order
        // every lane would start a row of its own) and each dword is then
        // moved to its fragment lane (q, r), which takes row r, piece q from
        // lane 4 r + q
        const uint16_t *w1l = a.w1 + (size_t)(lane >> 2) * C + 8 * (lane & 3);
        const int perm = (4 * r + q) * 4;  // ds_bpermute source address
        const uint16_t *w2l = a.w2 + (size_t)(o0 + tau_row(m)) * a.EC + 8 * h;
        float16v acc[PB];
#pragma unroll
        for (int pb = 0; pb < PB; pb++)
#pragma unroll
            for (int e = 0; e < 16; e++)
                acc[pb][e] = 0.0f;
        // W1 fragments stream through a ring of four groups held in
        // registers: stream step st is group st % NG of the wave's chunk
        // st / NG, loaded four steps before its products (across chunks)
        const int ncw = wv < NCH ? (NCH - wv + NW - 1) / NW : 0;
        const int steps = ncw * NG;
        u32x4 f0[KG][2], f1[KG][2], f2[KG][2], f3[KG][2];
        // (steps past the wave's last one reload its last group: every load
        // is unconditional, so the compiler's count of loads in flight stays
        // exact across the loop and it waits for one group, not all of them)
        auto load_step = [&](int st, u32x4(&f)[KG][2]) {
            const int sc = st < steps ? st : (steps > 0 ? steps - 1 : 0);
            const int ch = steps > 0 ? wv + NW * (sc / NG) : 0, g = sc % NG;
            const uint16_t *p = w1l + (size_t)ch * 32 * C + 32 * KG * g;
#pragma unroll
            for (int kk = 0; kk < KG; kk++)
#pragma unroll
                for (int mt = 0; mt < 2; mt++)
                    f[kk][mt] = *reinterpret_cast<const u32x4 *>(p + (size_t)16 * mt * C + 32 * kk);
        };
        // W2 fragments of a chunk (output rows o0 + tau(m), hidden 32 ch + 16 kk
        // + 8 h ..), loaded one chunk ahead into one of two register sets
        auto load_w2 = [&](int cn, u32x4(&w)[2]) {
            const int cc = cn < ncw ? cn : (ncw > 0 ? ncw - 1 : 0);
            const int ch = ncw > 0 ? wv + NW * cc : 0;
#pragma unroll
            for (int kk = 0; kk < 2; kk++)
                w[kk] = *reinterpret_cast<const u32x4 *>(w2l + ch * 32 + 16 * kk);
        };
        // the raw ring slots moved into fragment lanes (lane (q, r): row r, piece q)
        auto permute = [&](const u32x4(&f)[KG][2], u32x4(&fa)[KG][2]) {
#pragma unroll
            for (int kk = 0; kk < KG; kk++)
#pragma unroll
                for (int mt = 0; mt < 2; mt++)
#pragma unroll
                    for (int d = 0; d < 4; d++)
                        fa[kk][mt][d] = (uint32_t)__builtin_amdgcn_ds_bpermute(perm, (int)f[kk][mt][d]);
        };
        u32x4 wa[2], wb[2], pa[KG][2], pq[KG][2];
        load_step(0, f0);
        load_step(1, f1);
        load_step(2, f2);
        load_step(3, f3);
        load_w2(0, wa);
        // (the first ring groups and W2 fragments load during the depth-wise conv)

        // 1b. depth-wise conv; thread keeps channel chunk q and items
        // pl = tid / C8 + it * NT / C8 in registers, each tap read once from LDS
        {
            const int q = tid % C8, pad = a.k >> 1;
            int hr[IT], wc[IT], nb[IT];
            float acc[IT][8];
#pragma unroll
            for (int it = 0; it < IT; it++) {
                const int pl = tid / C8 + it * (NT / C8);
                const int pc = pl < a.P ? pl : 0;
                const int n = pc / a.HW, rem = pc - n * a.HW;
                hr[it] = rem / a.W;
                wc[it] = rem - hr[it] * a.W;
                nb[it] = n * a.HW;
#pragma unroll
                for (int e = 0; e < 8; e++)
                    acc[it][e] = 0.0f;
            }
            for (int i = 0; i < a.k; i++)
                for (int j = 0; j < a.k; j++) {
                    Pack8 wt;
                    wt.u = *reinterpret_cast<const u32x4 *>(smem + a.off_d +
                                                            ((uint32_t)(i * a.k + j) * C8 + (uint32_t)q) * 16);
                    float wf[8];
#pragma unroll
                    for (int e = 0; e < 4; e++) {
                        wf[2 * e] = T::lo(wt.w[e]);
                        wf[2 * e + 1] = T::hi(wt.w[e]);
                    }
#pragma unroll
                    for (int it = 0; it < IT; it++) {
                        const int pl = tid / C8 + it * (NT / C8);
                        if (pl >= a.P)
                            continue;  // (wave-uniform at C = 512)
                        const int hi = hr[it] + i - pad, wj = wc[it] + j - pad;
                        const bool ok = (unsigned)hi < (unsigned)a.H && (unsigned)wj < (unsigned)a.W;
                        const uint32_t ad = ok ? (uint32_t)(nb[it] + hi * a.W + wj) * XP + (uint32_t)q * 16 : a.off_zero;
                        Pack8 xv;
                        xv.u = *reinterpret_cast<const u32x4 *>(smem + ad);
#pragma unroll
                        for (int e = 0; e < 4; e++) {
                            acc[it][2 * e] = fmaf(T::lo(xv.w[e]), wf[2 * e], acc[it][2 * e]);
                            acc[it][2 * e + 1] = fmaf(T::hi(xv.w[e]), wf[2 * e + 1], acc[it][2 * e + 1]);
                        }
                    }
                }
            float sc[8], bi[8];
#pragma unroll
            for (int e = 0; e < 8; e++) {
                sc[e] = a.s0 ? a.s0[q * 8 + e] : 1.0f;
                bi[e] = a.b0 ? a.b0[q * 8 + e] : 0.0f;
            }
            __syncthreads();  // every thread is done with x and the taps: D and s1, b1 may overwrite them
            // s1, b1 of every hidden channel (fp32) over the x pixels, so that
            // the chunk loop reads them without a branch on null vectors
            float *s1l = reinterpret_cast<float *>(smem), *b1l = s1l + a.EC;
            for (int i = tid; i < a.EC; i += NT) {
                s1l[i] = a.s1 ? a.s1[i] : 1.0f;
                b1l[i] = a.b1 ? a.b1[i] : 0.0f;
            }
#pragma unroll
            for (int it = 0; it < IT; it++) {
                const int pl = tid / C8 + it * (NT / C8);
                u32x4 d;
#pragma unroll
                for (int e = 0; e < 4; e++)
                    d[e] = pl < a.P ? T::pack2(fmaf(acc[it][2 * e], sc[2 * e], bi[2 * e]),
                                               fmaf(acc[it][2 * e + 1], sc[2 * e + 1], bi[2 * e + 1]))
                                    : 0u;
                *reinterpret_cast<u32x4 *>(smem + a.off_d + (uint32_t)pl * DP + (uint32_t)q * 16) = d;
            }
        }
        __syncthreads();

        // 2. the wave's chunks (the ring and the first W2 fragments are in
        // flight); the first group is permuted and its slot refilled
        permute(f0, pa);
        load_step(4, f0);
        auto run_chunk = [&](int c, const u32x4(&w2c)[2], u32x4(&w2n)[2]) {
            const int ch = wv + NW * c;
            // s1, b1 of the lane's hidden values (hidden 32 ch + 16 mt + 4 q + i)
            const float *s1l = reinterpret_cast<const float *>(smem), *b1l = s1l + a.EC;
            float4v s1v[2], b1v[2];
#pragma unroll
            for (int mt = 0; mt < 2; mt++) {
                const int hr = ch * 32 + 16 * mt + 4 * q;
                s1v[mt] = *reinterpret_cast<const float4v *>(s1l + hr);
                b1v[mt] = *reinterpret_cast<const float4v *>(b1l + hr);
            }
            float4v hh[PB][2][2];  // [block][pixel half nt][hidden half mt]
#pragma unroll
            for (int pb = 0; pb < PB; pb++)
#pragma unroll
                for (int nt = 0; nt < 2; nt++)
#pragma unroll
                    for (int mt = 0; mt < 2; mt++)
                        hh[pb][nt][mt] = float4v{0.f, 0.f, 0.f, 0.f};
            auto mma_group = [&](int g, const u32x4(&fa)[KG][2]) {
#pragma unroll
                for (int kk = 0; kk < KG; kk++)
#pragma unroll
                    for (int pb = 0; pb < PB; pb++)
#pragma unroll
                        for (int nt = 0; nt < 2; nt++) {
                            const u32x4 bd = *reinterpret_cast<const u32x4 *>(
                                smem + dbase + (uint32_t)(32 * pb + 16 * nt) * DP + (uint32_t)(g * KG + kk) * 64);
#pragma unroll
                            for (int mt = 0; mt < 2; mt++)
                                hh[pb][nt][mt] = T::mfma(fa[kk][mt], bd, hh[pb][nt][mt]);
                        }
            };
            // four groups per pass (a runtime loop keeps the reads of D that
            // the scheduler hoists to one pass).  While group j's products
            // run, group j + 1's fragments are permuted into the other
            // buffer and their raw slot is refilled four groups ahead; the
            // order is pinned
#pragma unroll 1
            for (int g = 0; g < NG; g += 4) {
                const int st = c * NG + g;
                mma_group(g, pa);
                permute(f1, pq);
                load_step(st + 5, f1);
                __builtin_amdgcn_sched_barrier(0);
                mma_group(g + 1, pq);
                permute(f2, pa);
                load_step(st + 6, f2);
                __builtin_amdgcn_sched_barrier(0);
                mma_group(g + 2, pa);
                permute(f3, pq);
                load_step(st + 7, f3);
                __builtin_amdgcn_sched_barrier(0);
                mma_group(g + 3, pq);
                permute(f0, pa);
                load_step(st + 8, f0);
                __builtin_amdgcn_sched_barrier(0);
            }
            // the next chunk's W2 fragments, behind this chunk's ring refills
            load_w2(c + 1, w2n);
            // phi(s1 u + b1), rounded to the I/O dtype; the lane pair (l, l ^ 16)
            // trades quads so that each lane holds hidden 16 kk + 8 h .. + 7 of
            // its pixel m: the B operand of the projection
#pragma unroll
            for (int pb = 0; pb < PB; pb++) {
                uint32_t pk[2][2][2];  // [nt][mt][pair]
#pragma unroll
                for (int nt = 0; nt < 2; nt++)
#pragma unroll
                    for (int mt = 0; mt < 2; mt++)
#pragma unroll
                        for (int j = 0; j < 2; j++) {
                            const float u0 = act(fmaf(hh[pb][nt][mt][2 * j], s1v[mt][2 * j], b1v[mt][2 * j]), a.act);
                            const float u1 =
                                act(fmaf(hh[pb][nt][mt][2 * j + 1], s1v[mt][2 * j + 1], b1v[mt][2 * j + 1]), a.act);
                            pk[nt][mt][j] = T::pack2(u0, u1);
                        }
#pragma unroll
                for (int kk = 0; kk < 2; kk++) {
                    uint32_t own[2], rcv[2];
#pragma unroll
                    for (int j = 0; j < 2; j++) {
                        own[j] = b ? pk[1][kk][j] : pk[0][kk][j];
                        const uint32_t snd = b ? pk[0][kk][j] : pk[1][kk][j];
                        rcv[j] = (uint32_t)__shfl_xor((int)snd, 16);
                    }
                    const u32x4 hid =
                        b ? u32x4{rcv[0], rcv[1], own[0], own[1]} : u32x4{own[0], own[1], rcv[0], rcv[1]};
                    acc[pb] = mfma32(w2c[kk], hid, acc[pb], T{});
                }
            }
        };
        // two chunks per iteration, so the W2 register sets alternate without a copy
        int c = 0;
        for (; c + 1 < ncw; c += 2) {
            run_chunk(c, wa, wb);
            run_chunk(c + 1, wb, wa);
        }
        if (c < ncw)
            run_chunk(c, wa, wb);

        __syncthreads();  // every wave is done with s1, b1

        // 3. projections into the x area:
        // wave w, block pb, register quad g4 of lane l at float index
        // ((w * PB + pb) * 4 + g4) * 256 + 4 l; register e of lane (h, m) is
        // channel o0 + 16 h + e of pixel 32 pb + m
        float *red = reinterpret_cast<float *>(smem);
#pragma unroll
        for (int pb = 0; pb < PB; pb++)
#pragma unroll
            for (int g4 = 0; g4 < 4; g4++)
                *reinterpret_cast<float4v *>(red + ((wv * PB + pb) * 4 + g4) * 256 + 4 * lane) =
                    float4v{acc[pb][4 * g4], acc[pb][4 * g4 + 1], acc[pb][4 * g4 + 2], acc[pb][4 * g4 + 3]};
        __syncthreads();
        if (tid < PB * 256) {
            const int pb = tid >> 8, g4 = (tid >> 6) & 3, ln = tid & 63;
            float4v s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int w = 0; w < NW; w++) {
                const float4v v = *reinterpret_cast<const float4v *>(red + ((w * PB + pb) * 4 + g4) * 256 + 4 * ln);
#pragma unroll
                for (int e = 0; e < 4; e++)
                    s[e] += v[e];
            }
            const int p = 32 * pb + (ln & 31), c = o0 + 16 * (ln >> 5) + 4 * g4;
            if (p < a.P) {
                const u32x2 xv = *reinterpret_cast<const u32x2 *>(a.x + (size_t)p * C + c);
                float o[4];
#pragma unroll
                for (int e = 0; e < 4; e++) {
                    const float sv = a.s2 ? a.s2[c + e] : 1.0f, bv = a.b2 ? a.b2[c + e] : 0.0f;
                    const uint32_t xw = xv[e >> 1];
                    o[e] = ((e & 1) ? T::hi(xw) : T::lo(xw)) + fmaf(s[e], sv, bv);
                }
                *reinterpret_cast<u32x2 *>(a.y + (size_t)p * C + c) = u32x2{T::pack2(o[0], o[1]), T::pack2(o[2], o[3])};
            }
        }
    }
};

template <typename T, int C, int PB>
__global__ __launch_bounds__(NT, 1) void slice_kernel(Args a) {
    extern __shared__ __attribute__((aligned(256))) uint8_t smem[];
    Kern<T, C, PB>::run(a, smem);
}

// LDS layout: [x pixels | s1, b1 (fp32) | the waves' projections] [zero piece] [taps | D pixels]
struct Plan {
    int pb;
    uint32_t off_zero, off_d;
    size_t lds;
};

inline bool plan(const Shape &s, Plan &pl) {
    const int64_t P = (int64_t)s.N * s.H * s.W;
    if (P < 1 || P > PMAX || (s.C != 128 && s.C != 256 && s.C != 512) || (s.E * s.C) % 32 != 0 || s.k < 1 ||
        s.k > 7 || s.k % 2 == 0)
        return false;
    pl.pb = P <= 32 ? 1 : 2;
    const size_t npx = (size_t)pl.pb * 32;
    const size_t r0 = std::max(std::max(npx * s.C * 2, (size_t)NW * pl.pb * 4096), (size_t)s.E * s.C * 8);
    pl.off_zero = (uint32_t)((r0 + 255) & ~(size_t)255);
    pl.off_d = pl.off_zero + 256;
    // the D region first holds the taps [k][k][C]
    pl.lds = pl.off_d + std::max(npx * ((size_t)s.C * 2 + 16), (size_t)s.k * s.k * s.C * 2);
    return pl.lds <= 160 * 1024;
}

template <typename T, int C, int PB>
hipError_t launch_t(const Args &a, size_t lds, hipStream_t st) {
    auto kf = slice_kernel<T, C, PB>;
    hipError_t e = allow_full_lds((const void *)kf);
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(kf, dim3(C / 32), dim3(NT), lds, st, a);
    return hipGetLastError();
}

template <typename T>
hipError_t launch_c(const Args &a, int C, int pb, size_t lds, hipStream_t st) {
    switch (C * 2 + pb - 1) {
    case 256: return launch_t<T, 128, 1>(a, lds, st);
    case 257: return launch_t<T, 128, 2>(a, lds, st);
    case 512: return launch_t<T, 256, 1>(a, lds, st);
    case 513: return launch_t<T, 256, 2>(a, lds, st);
    case 1024: return launch_t<T, 512, 1>(a, lds, st);
    case 1025: return launch_t<T, 512, 2>(a, lds, st);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace slice

bool slice_applies(const Shape &s) {
    slice::Plan pl;
    return slice::plan(s, pl);
}

hipError_t launch_slice(const void *x, void *y, const BlockW &w, const Shape &s, hipStream_t st) {
    slice::Plan pl;
    if (!slice::plan(s, pl))
        return hipErrorInvalidConfiguration;
    slice::Args a{};
    a.x = (const uint16_t *)x;
    a.dw_w = (const uint16_t *)w.dw_w;
    a.w1 = (const uint16_t *)w.w1;
    a.w2 = (const uint16_t *)w.w2;
    a.s0 = w.s0;
    a.b0 = w.b0;
    a.s1 = w.s1;
    a.b1 = w.b1;
    a.s2 = w.s2;
    a.b2 = w.b2;
    a.y = (uint16_t *)y;
    a.H = s.H;
    a.W = s.W;
    a.HW = s.H * s.W;
    a.EC = s.E * s.C;
    a.k = s.k;
    a.act = s.act;
    a.P = s.N * s.H * s.W;
    a.off_zero = pl.off_zero;
    a.off_d = pl.off_d;
    return s.bf16 ? slice::launch_c<BF16>(a, s.C, pl.pb, pl.lds, st)
                  : slice::launch_c<F16>(a, s.C, pl.pb, pl.lds, st);
}

}  // namespace cf
