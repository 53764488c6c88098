// cf_small.hip -- hidden-split fused block for small batches (Sec. 5.3.1 with
// the channel partition of the hidden dimension over workgroups and global
// partial sums; the latency regime of Sec. 4.1.2, where the weights, not the
// activations, dominate the bytes).
//
// Grid: (tiles of at most TP pixels, hidden groups, output slices of 128).  One
// workgroup of 4 waves:
//  1. copies the input rows of its tile plus the k/2 halo rows into LDS
//     (in-image columns only; rows outside the batch are zero-filled; all
//     loads in flight before the first LDS write),
//  2. computes the depth-wise conv with one thread per (pixel, 8 channels)
//     into an LDS D buffer, d = s0 * conv + b0,
//  3. wave w takes pixels 32w .. 32w+31 of the tile: it reads its D columns
//     as MFMA B fragments, then for each hidden chunk of its group runs the
//     expand (W1 fragments from global memory into registers; for C = 512,
//     where a W1 row is one 1 KB copy, through LDS by LDS-DMA instead: the
//     first chunk beside the halo, later chunks through a two-slot ring in
//     the halo and D areas), phi(s1 * u + b1) in fp32, and the project onto
//     its output channels,
//  4. writes s2 * (its projection) as an fp32 partial; a second kernel adds
//     the groups' partials in order, b2 and x.  With a single group the
//     workgroup stores y = x + s2 * projection + b2 itself.
// The products use v_mfma_f32_32x32x16 with weights as the A operand (rows in
// the sigma / tau orders of cf_fused_impl.h) and pixels as the B operand.
#include "cf_device.h"
#include "cf_fused_impl.h"
#include "cf_kernels.h"

namespace cf {
namespace small {

using fused::mfma32;
using fused::sigma_row;
using fused::tau_row;
using fused::float16v;

constexpr int NT = 256;
constexpr int TPMAX = 128;  // pixels per tile (32 per wave)

struct Args {
    const uint16_t *x;
    const uint16_t *dw_w;
    const float *s0, *b0;
    const uint16_t *w1;
    const float *s1, *b1;
    const uint16_t *w2;
    const float *s2;
    float *partial;  // [groups][P][C]
    uint16_t *y;     // one hidden group: the block output itself (no partials)
    const float *b2;
    int H, W, NH, C, EC, act;
    uint32_t P;
    int tp;           // pixels per tile
    int halo_rows;    // LDS halo rows per tile
    int chunks_per_group;
    uint32_t off_d;     // LDS byte offset of the D buffer
    uint32_t off_zero;  // LDS byte offset of one zero pixel (taps outside the image read it)
    uint32_t off_s2;    // LDS byte offset of this output slice's s2 (fp32)
    uint32_t off_w1;    // C = 512: LDS byte offset of the first chunk's W1 rows (0: W1 from global memory)
    int ring;           // C = 512: later chunks' W1 through a two-slot LDS ring at offset 0 (0: registers)
    fused::FastDiv divW, divH;
};

template <typename T, int C, int KS>
struct Kern {
    static constexpr int PAD = KS / 2, KST = C / 16, C8 = C / 8;
    static constexpr int CO = C < 128 ? C : 128, OSPLIT = C / CO, CBO = CO / 32;  // output channels per workgroup
    static constexpr int PIXB = C * 2 + 16;  // LDS bytes per halo / D pixel
    static constexpr int HB = C == 512 ? 8 : 16;  // halo loads in flight per thread
    // request the first chunk's weights at kernel start (registers permitting)
    static constexpr bool PRELOAD = KS <= 3;
    // C = 512: a W1 row is 1 KB, one LDS-DMA instruction; rows sit W1P bytes
    // apart so that the 16 rows sigma(m) of a 16-lane fragment read fall in
    // 16 different bank groups
    static constexpr bool LW1 = C == 512;
    static constexpr uint32_t W1P = 1040;
    static constexpr uint32_t RSLOT = 32 * W1P;  // one chunk's W1 rows in the ring

    static __device__ void run(const Args &a, uint8_t *smem) {
        const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
        const int h = lane >> 5, m = lane & 31;
        const uint32_t p0 = blockIdx.x * (uint32_t)a.tp;
        uint32_t pend = p0 + (uint32_t)a.tp;
        if (pend > a.P)
            pend = a.P;
        const int WP = a.W;  // LDS columns: the image's own (taps outside it are skipped)
        const uint32_t g_lo = p0 / (uint32_t)a.W;  // first image row (over N*H) of the tile
        const int rows = a.halo_rows;
        const int ob = blockIdx.z;  // output half
        const int ch0 = blockIdx.y * a.chunks_per_group;

        // The first chunk's weight fragments and s1 / b1 are requested before
        // anything else, so their latency overlaps the halo copy and the
        // depth-wise conv (one wave per SIMD: the registers are there).
        u32x4 w1r[KST], w2r[2 * CBO];
        float s1r[16], b1r[16];
        auto load_chunk = [&](int ch, bool with_w1) {
            const uint16_t *w1p = a.w1 + (size_t)(ch * 32 + sigma_row(m)) * C + 8 * h;
            if (with_w1) {
#pragma unroll
                for (int ks = 0; ks < KST; ks++)
                    w1r[ks] = *reinterpret_cast<const u32x4 *>(w1p + 16 * ks);
            }
#pragma unroll
            for (int i = 0; i < 2 * CBO; i++) {
                const int cb = i >> 1, kk = i & 1;
                const int o = ob * CO + cb * 32 + tau_row(m);
                w2r[i] = *reinterpret_cast<const u32x4 *>(a.w2 + (size_t)o * a.EC + ch * 32 + 16 * kk + 8 * h);
            }
            // register e = 4t + i <-> hidden ch*32 + 16(t>>1) + 8h + 4(t&1) + i
#pragma unroll
            for (int e = 0; e < 16; e++) {
                const int t = e >> 2, i = e & 3;
                const int r = ch * 32 + 16 * (t >> 1) + 8 * h + 4 * (t & 1) + i;
                s1r[e] = a.s1 ? a.s1[r] : 1.0f;
                b1r[e] = a.b1 ? a.b1[r] : 0.0f;
            }
        };
        // C = 512 with room in LDS: the first chunk's W1 (32 KB, the same for
        // every wave) is copied once per workgroup, 1 KB per contiguous
        // LDS-DMA instruction, instead of being gathered four times into
        // registers; wave wv copies rows wv, wv + 4, ...
        const bool lw1 = LW1 && a.off_w1 != 0;
        if (lw1) {
            const uint16_t *src = a.w1 + (size_t)ch0 * 32 * C;
#pragma unroll
            for (int i = 0; i < 8; i++) {
                const int r = wv + 4 * i;
                fused::dma16s(src + (size_t)r * C, (uint32_t)lane * 16, smem + a.off_w1 + (uint32_t)r * W1P);
            }
        }
        if constexpr (PRELOAD)
            load_chunk(ch0, !lw1);

        // the zero pixel, and s2 of this output slice
        for (int i = tid; i < PIXB / 16; i += NT)
            *reinterpret_cast<u32x4 *>(smem + a.off_zero + i * 16) = u32x4{0u, 0u, 0u, 0u};
        for (int i = tid; i < CO; i += NT)
            reinterpret_cast<float *>(smem + a.off_s2)[i] = a.s2 ? a.s2[ob * CO + i] : 1.0f;

        // 1. halo rows g_lo - PAD .. into LDS, padded pixels zero
        {
            const int total = rows * WP * C8;
            for (int c0 = 0; c0 < total; c0 += HB * NT) {
                u32x4 v[HB];
                int dst[HB];
#pragma unroll
                for (int u = 0; u < HB; u++) {
                    const int ci = c0 + u * NT + tid;
                    const int r = ci / (WP * C8), rem = ci - r * (WP * C8);
                    const int col = rem / C8, q = rem - col * C8;
                    const int px = col, grow = (int)g_lo - PAD + r;
                    dst[u] = ci < total ? (r * WP + col) * PIXB + q * 16 : -1;
                    v[u] = u32x4{0u, 0u, 0u, 0u};
                    if (ci < total && px >= 0 && px < a.W && grow >= 0 && grow < a.NH)
                        v[u] = *reinterpret_cast<const u32x4 *>(a.x + ((size_t)grow * a.W + px) * C + q * 8);
                }
#pragma unroll
                for (int u = 0; u < HB; u++)
                    if (dst[u] >= 0)
                        *reinterpret_cast<u32x4 *>(smem + dst[u]) = v[u];
            }
        }
        __syncthreads();

        // 2. depth-wise conv: item = (pixel of the tile, 8 channels); NT is a
        // multiple of C/8, so a thread always works on the same channel chunk
        // q and holds its taps, s0 and b0 in registers.  A tap outside the
        // pixel's image reads the zero pixel, so the reads of a kernel row
        // carry no branch and are issued ahead of its FMAs (one wave per
        // SIMD: nothing else hides their latency).
        {
            const int q = tid % C8;
            constexpr bool TF = KS <= 3;  // taps as fp32 and branch-free reads (registers permitting)
            Pack8 wt[KS * KS];
#pragma unroll
            for (int t = 0; t < KS * KS; t++)
                wt[t].u = *reinterpret_cast<const u32x4 *>(a.dw_w + (size_t)t * C + q * 8);
            float wtf[TF ? KS * KS : 1][8];
            if constexpr (TF) {
#pragma unroll
                for (int t = 0; t < KS * KS; t++)
#pragma unroll
                    for (int e = 0; e < 4; e++) {
                        wtf[t][2 * e] = T::lo(wt[t].w[e]);
                        wtf[t][2 * e + 1] = T::hi(wt[t].w[e]);
                    }
            }
            float sc[8], bi[8];
#pragma unroll
            for (int e = 0; e < 8; e++) {
                sc[e] = a.s0 ? a.s0[q * 8 + e] : 1.0f;
                bi[e] = a.b0 ? a.b0[q * 8 + e] : 0.0f;
            }
            if constexpr (TF) {
                const uint32_t zaddr = a.off_zero + (uint32_t)q * 16;
                for (int pl = tid / C8; pl < a.tp; pl += NT / C8) {
                    const uint32_t p = p0 + pl;
                    const bool pv = p < a.P;
                    const uint32_t pc = pv ? p : p0;
                    const uint32_t gg = fused::fdiv(pc, a.divW);
                    const int wc = (int)(pc - gg * (uint32_t)a.W);
                    const int hr = (int)(gg - fused::fdiv(gg, a.divH) * (uint32_t)a.H);
                    float acc[8];
    #pragma unroll
                    for (int e = 0; e < 8; e++)
                        acc[e] = 0.0f;
    #pragma unroll
                    for (int i = 0; i < KS; i++) {
                        const int hi = hr + i - PAD;  // rows of another image or outside the batch: zero padding
                        const bool rok = pv && hi >= 0 && hi < a.H;
                        const int r = (int)(gg - g_lo) + i;
                        Pack8 xv[KS];
    #pragma unroll
                        for (int j = 0; j < KS; j++) {
                            const int wj = wc + j - PAD;
                            const bool ok = rok && wj >= 0 && wj < a.W;
                            const uint32_t ad = ok ? (uint32_t)((r * WP + wj) * PIXB + q * 16) : zaddr;
                            xv[j].u = *reinterpret_cast<const u32x4 *>(smem + ad);
                        }
    #pragma unroll
                        for (int j = 0; j < KS; j++)
    #pragma unroll
                            for (int e = 0; e < 4; e++) {
                                const float w0 = TF ? wtf[TF ? i * KS + j : 0][2 * e] : T::lo(wt[i * KS + j].w[e]);
                                const float w1 = TF ? wtf[TF ? i * KS + j : 0][2 * e + 1] : T::hi(wt[i * KS + j].w[e]);
                                acc[2 * e] = fmaf(T::lo(xv[j].w[e]), w0, acc[2 * e]);
                                acc[2 * e + 1] = fmaf(T::hi(xv[j].w[e]), w1, acc[2 * e + 1]);
                            }
                    }
                    u32x4 d;
    #pragma unroll
                    for (int e = 0; e < 4; e++)
                        d[e] = pv ? T::pack2(fmaf(acc[2 * e], sc[2 * e], bi[2 * e]),
                                             fmaf(acc[2 * e + 1], sc[2 * e + 1], bi[2 * e + 1]))
                                  : 0u;
                    *reinterpret_cast<u32x4 *>(smem + a.off_d + pl * PIXB + q * 16) = d;
                }
            } else {
                // k >= 5: the taps stay packed and rows outside the image are
                // skipped (registers do not allow every read of a pixel ahead)
                for (int pl = tid / C8; pl < a.tp; pl += NT / C8) {
                    const uint32_t p = p0 + pl;
                    float acc[8];
    #pragma unroll
                    for (int e = 0; e < 8; e++)
                        acc[e] = 0.0f;
                    if (p < a.P) {
                        const uint32_t gg = p / (uint32_t)a.W;
                        const int wc = (int)(p - gg * (uint32_t)a.W);
                        const int hr = (int)(gg % (uint32_t)a.H);
    #pragma unroll
                        for (int i = 0; i < KS; i++) {
                            const int hi = hr + i - PAD;
                            if (hi < 0 || hi >= a.H)
                                continue;  // rows of another image: zero padding
                            const int r = (int)(gg - g_lo) + i;
    #pragma unroll
                            for (int j = 0; j < KS; j++) {
                                const int wj = wc + j - PAD;
                                if (wj < 0 || wj >= a.W)
                                    continue;  // zero padding
                                Pack8 xv;
                                xv.u = *reinterpret_cast<const u32x4 *>(smem + (r * WP + wj) * PIXB + q * 16);
    #pragma unroll
                                for (int e = 0; e < 4; e++) {
                                    acc[2 * e] = fmaf(T::lo(xv.w[e]), T::lo(wt[i * KS + j].w[e]), acc[2 * e]);
                                    acc[2 * e + 1] = fmaf(T::hi(xv.w[e]), T::hi(wt[i * KS + j].w[e]), acc[2 * e + 1]);
                                }
                            }
                        }
                    }
                    u32x4 d;
    #pragma unroll
                    for (int e = 0; e < 4; e++)
                        d[e] = p < a.P ? T::pack2(fmaf(acc[2 * e], sc[2 * e], bi[2 * e]),
                                                  fmaf(acc[2 * e + 1], sc[2 * e + 1], bi[2 * e + 1]))
                                       : 0u;
                    *reinterpret_cast<u32x4 *>(smem + a.off_d + pl * PIXB + q * 16) = d;
                }
            }
        }
        if (lw1)
            fused::wait_vmcnt<0>();  // this wave's W1 copies have landed (published by the barrier)
        __syncthreads();

        // 3. this wave's pixels as B fragments: lane (h, m) = channels 16 ks + 8 h .. of pixel 32 wv + m
        const int pl = 32 * wv + m;
        // C = 512 with several chunks per group: once every wave holds its D
        // fragments the halo and D areas are no longer read, and they hold a
        // two-slot ring of W1 chunks copied by contiguous LDS-DMA (32 KB per
        // chunk once per workgroup, instead of gathered by each wave).  Every
        // wave then takes part in the copies and barriers, pixels or not.
        const bool ring = LW1 && a.ring != 0;
        const int nchg = a.chunks_per_group;
        auto issue_ring = [&](int ch, int slot) {
            const uint16_t *src = a.w1 + (size_t)ch * 32 * C;
#pragma unroll
            for (int i = 0; i < 8; i++) {
                const int r = wv + 4 * i;
                fused::dma16s(src + (size_t)r * C, (uint32_t)lane * 16, smem + (uint32_t)slot * RSLOT + (uint32_t)r * W1P);
            }
        };
        if (!ring && 32 * wv >= a.tp)
            return;  // no pixels for this wave (no barrier follows)
        if constexpr (!PRELOAD)
            load_chunk(ch0, !lw1);
        if (lw1) {
            // fragment (ks, lane h, m) = W1 row sigma(m), halves 16 ks + 8 h ..
            const uint8_t *w1l = smem + a.off_w1 + (uint32_t)sigma_row(m) * W1P + 16 * h;
#pragma unroll
            for (int ks = 0; ks < KST; ks++)
                w1r[ks] = *reinterpret_cast<const u32x4 *>(w1l + 32 * ks);
        }
        u32x4 dfr[KST];
#pragma unroll
        for (int ks = 0; ks < KST; ks++)
            dfr[ks] = pl < a.tp ? *reinterpret_cast<const u32x4 *>(smem + a.off_d + pl * PIXB + (16 * ks + 8 * h) * 2)
                                : u32x4{0u, 0u, 0u, 0u};

        if (ring) {
            __syncthreads();  // every wave holds its D fragments: halo and D areas free
            if (nchg > 1)
                issue_ring(ch0 + 1, 0);  // chunk j >= 1 goes to slot (j - 1) & 1
        }

        float16v acc[CBO];
#pragma unroll
        for (int c = 0; c < CBO; c++)
#pragma unroll
            for (int e = 0; e < 16; e++)
                acc[c][e] = 0.0f;

        for (int ch = ch0; ch < ch0 + nchg; ch++) {
            const int j = ch - ch0;
            if (ring && j >= 1) {
                fused::wait_vmcnt<0>();  // this wave's copies of chunk j (and its W2, s1, b1) landed
                __syncthreads();         // chunk j visible; chunk j - 1's slot free
                if (j + 1 < nchg)
                    issue_ring(ch + 1, j & 1);
                const uint8_t *w1l = smem + (uint32_t)((j - 1) & 1) * RSLOT + (uint32_t)sigma_row(m) * W1P + 16 * h;
#pragma unroll
                for (int ks = 0; ks < KST; ks++)
                    w1r[ks] = *reinterpret_cast<const u32x4 *>(w1l + 32 * ks);
            }
            float16v hh;
#pragma unroll
            for (int e = 0; e < 16; e++)
                hh[e] = 0.0f;
#pragma unroll
            for (int ks = 0; ks < KST; ks++)
                hh = mfma32(w1r[ks], dfr[ks], hh, T{});
            // phi(s1 u + b1)
            uint32_t g[8];
#pragma unroll
            for (int q = 0; q < 8; q++) {
                float v2[2];
#pragma unroll
                for (int z = 0; z < 2; z++) {
                    const int e = 2 * q + z;
                    float u = fmaf(hh[e], s1r[e], b1r[e]);
                    if (a.act == ACT_GELU)
                        u = gelu_f32(u);
                    else if (a.act == ACT_RELU)
                        u = fmaxf(u, 0.0f);
                    v2[z] = u;
                }
                g[q] = T::pack2(v2[0], v2[1]);
            }
            // project: K step kk of the chunk = hidden 16 kk .. 16 kk + 15
#pragma unroll
            for (int i = 0; i < 2 * CBO; i++) {
                const int cb = i >> 1, kk = i & 1;
                const u32x4 hid = {g[4 * kk], g[4 * kk + 1], g[4 * kk + 2], g[4 * kk + 3]};
                acc[cb] = mfma32(w2r[i], hid, acc[cb], T{});
            }
            if (ch + 1 < ch0 + nchg)
                load_chunk(ch + 1, !ring);
        }

        // 4. partial = s2 * projection: register e of acc[cb] <-> channel ob*CO + cb*32 + 16h + e.
        // With one hidden group and an output pointer the projection is the
        // whole sum: y = x + s2 * projection + b2, rounded, is stored instead.
        const uint32_t p = p0 + pl;
        if (a.y && pl < a.tp && p < a.P) {
#pragma unroll
            for (int cb = 0; cb < CBO; cb++) {
                const int cl = cb * 32 + 16 * h, c = ob * CO + cl;  // 16 channels c .. c + 15
                const uint16_t *xp = a.x + (size_t)p * C + c;
                Pack8 xv[2];
                xv[0].u = *reinterpret_cast<const u32x4 *>(xp);
                xv[1].u = *reinterpret_cast<const u32x4 *>(xp + 8);
                u32x4 o[2];
#pragma unroll
                for (int hv = 0; hv < 2; hv++)
#pragma unroll
                    for (int q = 0; q < 4; q++) {
                        const int e0 = 8 * hv + 2 * q;
                        const float *s2l = reinterpret_cast<const float *>(smem + a.off_s2) + cl + e0;
                        const float bb0 = a.b2 ? a.b2[c + e0] : 0.0f, bb1 = a.b2 ? a.b2[c + e0 + 1] : 0.0f;
                        o[hv][q] = T::pack2(T::lo(xv[hv].w[q]) + fmaf(acc[cb][e0], s2l[0], bb0),
                                            T::hi(xv[hv].w[q]) + fmaf(acc[cb][e0 + 1], s2l[1], bb1));
                    }
                uint16_t *yp = a.y + (size_t)p * C + c;
                *reinterpret_cast<u32x4 *>(yp) = o[0];
                *reinterpret_cast<u32x4 *>(yp + 8) = o[1];
            }
        } else if (pl < a.tp && p < a.P) {
            float *dst = a.partial + ((size_t)blockIdx.y * a.P + p) * C + ob * CO;
#pragma unroll
            for (int cb = 0; cb < CBO; cb++) {
#pragma unroll
                for (int q = 0; q < 4; q++) {
                    const int c = cb * 32 + 16 * h + 4 * q;
                    const float4v s2v = *reinterpret_cast<const float4v *>(smem + a.off_s2 + c * 4);
                    float4v v;
#pragma unroll
                    for (int e = 0; e < 4; e++)
                        v[e] = acc[cb][4 * q + e] * s2v[e];
                    *reinterpret_cast<float4v *>(dst + c) = v;
                }
            }
        }
    }
};

template <typename T, int C, int KS>
__global__ __launch_bounds__(NT, 1) void small_kernel(Args a) {
    extern __shared__ __attribute__((aligned(256))) uint8_t smem[];
    Kern<T, C, KS>::run(a, smem);
}

template <typename T, int C, int KS>
hipError_t launch_tk(Args a, int tiles, int groups, size_t lds, hipStream_t st) {
    auto kf = small_kernel<T, C, KS>;
    hipError_t e = allow_full_lds((const void *)kf);
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(kf, dim3(tiles, groups, Kern<T, C, KS>::OSPLIT), dim3(NT), lds, st, a);
    return hipGetLastError();
}

template <typename T, int C>
hipError_t launch_tc(Args a, int k, int tiles, int groups, size_t lds, hipStream_t st) {
    switch (k) {
    case 1: return launch_tk<T, C, 1>(a, tiles, groups, lds, st);
    case 3: return launch_tk<T, C, 3>(a, tiles, groups, lds, st);
    case 5: return launch_tk<T, C, 5>(a, tiles, groups, lds, st);
    case 7: return launch_tk<T, C, 7>(a, tiles, groups, lds, st);
    default: return hipErrorInvalidValue;
    }
}

template <typename T>
hipError_t launch_t(Args a, int k, int tiles, int groups, size_t lds, hipStream_t st) {
    switch (a.C) {
    case 64: return launch_tc<T, 64>(a, k, tiles, groups, lds, st);
    case 128: return launch_tc<T, 128>(a, k, tiles, groups, lds, st);
    case 256: return launch_tc<T, 256>(a, k, tiles, groups, lds, st);
    case 512: return launch_tc<T, 512>(a, k, tiles, groups, lds, st);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace small

// Tile plan of the small-batch kernel: pixels per tile, halo rows, LDS offsets.
struct SmallPlan {
    int tp, tiles, halo_rows;
    size_t off_d, off_zero, off_s2, off_w1, lds;
};

// false when the kernel does not apply (partials for more than 8 tiles, or no
// tile fits the LDS).  Writing y directly (one group, no partials), a tile may
// shrink below 128 pixels in steps of 32 until its halo and D buffer fit; the
// waves left without pixels idle.
static bool small_plan(const Shape &s, bool direct, SmallPlan &pl) {
    if (s.C != 64 && s.C != 128 && s.C != 256 && s.C != 512)
        return false;
    const int64_t P = (int64_t)s.N * s.H * s.W;
    int tp = P < small::TPMAX ? (int)P : small::TPMAX;
    for (;;) {
        const int64_t tiles = (P + tp - 1) / tp;
        if ((!direct && tiles > 8) || tiles > ((int64_t)1 << 30))
            return false;
        // image rows a tile of tp consecutive pixels touches, plus the halo
        int64_t span = (int64_t)(tp - 1) / s.W + 2;
        if (span > (int64_t)s.N * s.H)
            span = (int64_t)s.N * s.H;
        const int halo_rows = (int)span + 2 * (s.k / 2);
        const size_t pixb = (size_t)s.C * 2 + 16;
        pl.off_d = (((size_t)halo_rows * s.W * pixb) + 255) & ~(size_t)255;
        pl.off_zero = pl.off_d + (size_t)tp * pixb;
        pl.off_s2 = pl.off_zero + pixb;
        const size_t co = s.C < 128 ? (size_t)s.C : 128;
        pl.lds = pl.off_s2 + co * 4;
        if (pl.lds <= 160 * 1024) {
            pl.tp = tp;
            pl.tiles = (int)tiles;
            pl.halo_rows = halo_rows;
            break;
        }
        if (!direct || tp <= 32)
            return false;
        tp = ((tp - 1) / 32) * 32;  // next smaller multiple of 32
    }
    // C = 512: the first chunk's W1 rows through LDS when they fit beside the rest
    pl.off_w1 = 0;
    if (s.C == 512) {
        const size_t o = (pl.lds + 15) & ~(size_t)15;
        if (o + 32 * (size_t)1040 <= 160 * 1024) {
            pl.off_w1 = o;
            pl.lds = o + 32 * (size_t)1040;
        }
    }
    return true;
}

// LDS bytes the small-batch kernel needs for this shape, 0 if it does not apply
// (the C = 512 launch adds the first chunk's W1 rows when they still fit).
size_t small_split_lds_bytes(const Shape &s, bool direct) {
    SmallPlan pl;
    return small_plan(s, direct, pl) ? pl.lds : 0;
}

// Small-batch hidden-split path: partial[g][P][C] = s2 * (W2 phi(s1 W1 D + b1))
// restricted to the chunks of group g, or with groups = 1 and y non-null
// y = x + s2 * (W2 phi(s1 W1 D + b1)) + b2.  Returns hipErrorInvalidConfiguration
// when the shape does not suit it (partials for more than 8 tiles of 128
// pixels, or no tile whose halo and D buffer fit the LDS).  Writing y
// directly, every workgroup owns one tile, so any number of tiles works.
hipError_t launch_small_split(const void *x, const BlockW &w, const Shape &s, int groups, float *partial,
                              hipStream_t st, void *y) {
    if (y && groups != 1)
        return hipErrorInvalidValue;
    SmallPlan pl;
    if (!small_plan(s, y != nullptr, pl))
        return hipErrorInvalidConfiguration;
    const int64_t P = (int64_t)s.N * s.H * s.W;
    const int tp = pl.tp, tiles = pl.tiles, halo_rows = pl.halo_rows;
    const size_t off_d = pl.off_d, off_zero = pl.off_zero, off_s2 = pl.off_s2, off_w1 = pl.off_w1, lds = pl.lds;
    small::Args a{};
    a.x = (const uint16_t *)x;
    a.dw_w = (const uint16_t *)w.dw_w;
    a.s0 = w.s0;
    a.b0 = w.b0;
    a.w1 = (const uint16_t *)w.w1;
    a.s1 = w.s1;
    a.b1 = w.b1;
    a.w2 = (const uint16_t *)w.w2;
    a.s2 = w.s2;
    a.partial = partial;
    a.y = (uint16_t *)y;
    a.b2 = w.b2;
    a.H = s.H;
    a.W = s.W;
    a.NH = s.N * s.H;
    a.C = s.C;
    a.EC = s.E * s.C;
    a.act = s.act;
    a.P = (uint32_t)P;
    a.tp = tp;
    a.halo_rows = halo_rows;
    a.chunks_per_group = s.E * s.C / 32 / groups;
    a.off_d = (uint32_t)off_d;
    a.off_zero = (uint32_t)off_zero;
    a.off_s2 = (uint32_t)off_s2;
    a.off_w1 = (uint32_t)off_w1;
    a.ring = (s.C == 512 && a.chunks_per_group > 1 && off_zero >= 2 * (size_t)32 * 1040) ? 1 : 0;
    a.divW = fused::make_fastdiv((uint32_t)s.W);
    a.divH = fused::make_fastdiv((uint32_t)s.H);
    return s.bf16 ? small::launch_t<BF16>(a, s.k, tiles, groups, lds, st)
                  : small::launch_t<F16>(a, s.k, tiles, groups, lds, st);
}

}  // namespace cf
