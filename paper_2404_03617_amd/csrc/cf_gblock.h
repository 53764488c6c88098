// cf_gblock.h -- fused ConvFirst block with the paper's own first layer: a
// 3 x 3 grouped convolution of group width 8 (Sec. 5.3 of Lavin,
// arXiv:2404.03617, eq. f:grouped-conv2d with K = C, T = 8), then the FFN
// (expand, activation, project) in the loop-fused order of eq. e:ffn-eff, and
// the residual shortcut; batch norms folded to per-channel scale and bias.
// Instantiated per channel count in cf_gblock_c*.hip.
//
// Work unit: a block of 2 image rows x 16 columns (32 pixels) of one image.
// A workgroup of NW waves runs NW blocks at a time, one per wave; waves share
// the FFN weights, which stream through a two-slot LDS ring one chunk of 32
// hidden channels at a time (one workgroup barrier per chunk), and keep their
// own halo (4 rows x 18 columns) in a private LDS region.
//
// All products are v_mfma_f32_16x16x32 (fp16 or bf16 in, fp32 accumulate).
// Layouts (lane l, q = l >> 4, j = l & 15): A row j, k = 8q..8q+7; B column j,
// k = 8q..8q+7; D column j, rows 4q..4q+3.
//
//  * Grouped conv on the matrix unit.  For group g (channels 8g..8g+7) one
//    16 x 16 x 32 product per tap column dj evaluates 16 output pixels x 2
//    rows at once: D row m = 8s + o is output channel 8g + o of block row s,
//    D column j is block column j, and the K index is (tap row R of the
//    4-row halo window, input channel t) -- B lane (j, q) reads halo pixel
//    (row q, column j + dj), channels 8g..8g+7, one 16-byte LDS read; A row
//    (s, o) at (R, t) is the tap W[R - s][dj][8g + o][t], zero when R - s is
//    outside 0..2.  Three products per group cover the 3 x 3 taps; 72 of
//    every 96 multiply-adds are useful (a block-diagonal product with 16
//    output channels and 16 input channels per step would use 50% or less).
//  * The conv output d = s0 * conv + b0, rounded to the I/O dtype, goes to the
//    wave's LDS region (it overlays the halo, which the wave has finished
//    reading) and comes back as the expand's B fragments, read once per
//    block and kept in registers for every hidden chunk.
//  * Expand: two 16-row products per chunk and K step, with the W1 rows of a
//    chunk ordered so that expand tile t row m is hidden channel
//    8 (m >> 2) + 4 t + (m & 3): lane group q then holds hidden channels
//    8q..8q+7 -- exactly the B fragment of the project product, which needs
//    no data movement.  s1, b1 and the activation are applied in fp32, the
//    result rounded to the I/O dtype.
//  * Project: C/16 products per chunk into fp32 accumulators; the epilogue
//    adds s2, b2 and the block input x (re-read from global memory, an L2
//    hit) and stores the output once.
//  * The next block's halo is loaded during the FFN, a few 16-byte pieces per
//    lane per chunk, into the wave's region (free once the D fragments are in
//    registers).  Pixels outside the image are stored as zeros.
#pragma once
#include "cf_device.h"
#include "cf_fused_impl.h"
#include "cf_kernels.h"

namespace cf {
namespace gblk {

using fused::FastDiv;
using fused::fdiv;

constexpr int GW = 8;               // group width of the grouped conv
constexpr int BR = 2, BC = 16;      // block: 2 rows x 16 columns
constexpr int HR = BR + 2, HC = BC + 2;
constexpr int HPIX = HR * HC;       // halo pixels of a block (3 x 3 taps)
constexpr int HSTEP = 4;            // halo pieces per lane per FFN chunk

struct Args {
    const uint16_t *x;
    uint16_t *y;
    const uint16_t *gw;             // [3][3][C][8]
    const float *s0, *b0;
    const uint16_t *w1;             // [EC][C]
    const float *s1, *b1;
    const uint16_t *w2;             // [C][EC]
    const float *s2, *b2;
    int H, W, EC;
    int nch;                        // chunks of 32 hidden channels, ceil(EC / 32)
    int RP, SEG;                    // row pairs ceil(H/2), 16-column segments ceil(W/16)
    int nblocks;                    // N * RP * SEG
    int rbase, rextra;              // rounds (NW blocks) per workgroup: rbase, +1 for the first rextra
    int xcd_map;                    // 1: workgroup i takes range (i % 8) * (G / 8) + i / 8
};

__device__ __forceinline__ u32x4 lds16(const uint8_t *base, uint32_t off) {
    return *reinterpret_cast<const u32x4 *>(base + off);
}
__device__ __forceinline__ void sts16(uint8_t *base, uint32_t off, const u32x4 &v) {
    *reinterpret_cast<u32x4 *>(base + off) = v;
}

template <int C, int NW, typename T, int ACT>
struct GB {
    static_assert(C % 16 == 0 && C >= 16, "C must be a multiple of 16");
    static constexpr int NT = NW * 64;
    static constexpr int PB = 2 * C + 16;          // LDS bytes per pixel (odd multiple of 16)
    static constexpr int C8 = C / 8;               // 16-byte pieces per pixel
    static constexpr int NG = C / GW;              // groups
    static constexpr int KST = (C + 31) / 32;      // expand K steps of 32 channels
    static constexpr int MO = C / 16;              // project tiles of 16 output channels
    static constexpr int HALO = HPIX * PB;         // a wave's LDS region
    static constexpr int W1B = 2 * KST * 1024;     // chunk: W1 fragments
    static constexpr int W2B = MO * 1024;          //        W2 fragments
    static constexpr int CHB = W1B + W2B + 256;    //        then s1[32], b1[32]
    static constexpr int GROW = 3 * C * 16 + 128;  // conv taps of one tap row (+128: conflict-free)
    static constexpr int OFF_VEC = 3 * GROW;                  // s0, b0, s2, b2: C floats each
    static constexpr int OFF_RING = (OFF_VEC + 16 * C + 255) & ~255;
    static constexpr int OFF_HALO = OFF_RING + 2 * CHB;
    static constexpr int LDS = OFF_HALO + NW * HALO;
    static constexpr int HPIECES = HPIX * C8;      // 16-byte pieces of a halo
    static constexpr int HSTEPS = (HPIECES + 64 * HSTEP - 1) / (64 * HSTEP);
    static constexpr int CPIECES = (2 * KST + MO) * 64 + 16;
    static constexpr int CPT = (CPIECES + NT - 1) / NT;
    static_assert(LDS <= 160 * 1024, "LDS plan exceeds 160 KB");

    // ---- one chunk of FFN weights, fragment order, staged through registers
    static __device__ __forceinline__ void chunk_load(const Args &a, int ch, int tid, u32x4 (&r)[CPT]) {
#pragma unroll
        for (int u = 0; u < CPT; u++) {
            const int p = u * NT + tid;
            u32x4 v = {0u, 0u, 0u, 0u};
            if (p < 2 * KST * 64) {
                const int f = p >> 6, ln = p & 63, t = f / KST, kk = f - t * KST;
                const int m = ln & 15, qq = ln >> 4;
                const int row = ch * 32 + 8 * (m >> 2) + 4 * t + (m & 3);
                const int col = 32 * kk + 8 * qq;
                if (row < a.EC && col < C)
                    v = *reinterpret_cast<const u32x4 *>(a.w1 + (size_t)row * C + col);
            } else if (p < (2 * KST + MO) * 64) {
                const int pp = p - 2 * KST * 64;
                const int mo = pp >> 6, ln = pp & 63;
                const int o = 16 * mo + (ln & 15), hc = ch * 32 + 8 * (ln >> 4);
                if (hc < a.EC)
                    v = *reinterpret_cast<const u32x4 *>(a.w2 + (size_t)o * a.EC + hc);
            } else if (p < CPIECES) {
                const int jv = p - (2 * KST + MO) * 64;  // 0..7: s1, 8..15: b1
                const int hid = ch * 32 + 4 * (jv & 7);
                float4v f = {0.f, 0.f, 0.f, 0.f};
                if (hid < a.EC) {
                    const float *src = jv < 8 ? a.s1 : a.b1;
                    if (src)
                        f = *reinterpret_cast<const float4v *>(src + hid);
                    else if (jv < 8)
                        f = float4v{1.f, 1.f, 1.f, 1.f};
                }
                v = __builtin_bit_cast(u32x4, f);
            }
            r[u] = v;
        }
    }
    static __device__ __forceinline__ void chunk_store(uint8_t *slot, int tid, const u32x4 (&r)[CPT]) {
#pragma unroll
        for (int u = 0; u < CPT; u++) {
            const int p = u * NT + tid;
            if (p < CPIECES)
                sts16(slot, (uint32_t)p * 16, r[u]);
        }
    }

    // ---- block geometry
    struct Blk {
        int n, r0, c0;  // image, first row, first column
        bool valid;
    };
    static __device__ __forceinline__ Blk decode(const Args &a, int b) {
        Blk k;
        k.valid = b < a.nblocks;
        const int bb = k.valid ? b : 0;
        const int seg = bb % a.SEG, t = bb / a.SEG;
        const int rp = t % a.RP;
        k.n = t / a.RP;
        k.r0 = 2 * rp;
        k.c0 = 16 * seg;
        return k;
    }

    // halo piece i of block k: global source (or null for a zero pixel) and
    // LDS offset within the wave's region
    static __device__ __forceinline__ u32x4 halo_piece(const Args &a, const Blk &k, int i, uint32_t &dst) {
        const int px = i / C8, cq = i - px * C8;
        const int r = px / HC, cc = px - r * HC;
        const int h = k.r0 - 1 + r, w = k.c0 - 1 + cc;
        dst = (uint32_t)px * PB + (uint32_t)cq * 16;
        u32x4 v = {0u, 0u, 0u, 0u};
        if (k.valid && h >= 0 && h < a.H && w >= 0 && w < a.W)
            v = *reinterpret_cast<const u32x4 *>(a.x + (((size_t)k.n * a.H + h) * a.W + w) * C + 8 * cq);
        return v;
    }
    static __device__ __forceinline__ void halo_step_load(const Args &a, const Blk &k, int step, int lane,
                                                          u32x4 (&v)[HSTEP], uint32_t (&d)[HSTEP]) {
#pragma unroll
        for (int u = 0; u < HSTEP; u++) {
            const int i = (step * HSTEP + u) * 64 + lane;
            d[u] = 0xffffffffu;
            v[u] = u32x4{0u, 0u, 0u, 0u};
            if (i < HPIECES)
                v[u] = halo_piece(a, k, i, d[u]);
        }
    }
    static __device__ __forceinline__ void halo_step_store(uint8_t *reg, const u32x4 (&v)[HSTEP],
                                                           const uint32_t (&d)[HSTEP]) {
#pragma unroll
        for (int u = 0; u < HSTEP; u++)
            if (d[u] != 0xffffffffu)
                sts16(reg, d[u], v[u]);
    }

    static __device__ __forceinline__ float act(float u) {
        if constexpr (ACT == ACT_RELU)
            return fmaxf(u, 0.0f);
        else if constexpr (ACT == ACT_GELU)
            return gelu_f32(u);
        else
            return u;
    }

    static __device__ void run(const Args &a, uint8_t *smem) {
        const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
        const int q = lane >> 4, jl = lane & 15;
        const int G = gridDim.x;
        const int gi = a.xcd_map ? (int)(blockIdx.x % 8) * (G / 8) + (int)(blockIdx.x / 8) : (int)blockIdx.x;
        const int nr = a.rbase + (gi < a.rextra ? 1 : 0);
        const int rstart = gi * a.rbase + (gi < a.rextra ? gi : a.rextra);
        if (nr == 0)
            return;  // uniform over the workgroup, before any barrier

        uint8_t *gwl = smem;
        uint8_t *ring = smem + OFF_RING;
        uint8_t *reg = smem + OFF_HALO + wv * HALO;

        // grouped-conv taps: tap row i at i * GROW, then (column, channel) x 16 B
        for (int i = tid; i < 9 * C; i += NT) {
            const int tap = i / C, c = i - tap * C;
            sts16(gwl, (uint32_t)(tap / 3) * GROW + (uint32_t)((tap % 3) * C + c) * 16,
                  *reinterpret_cast<const u32x4 *>(a.gw + ((size_t)tap * C + c) * GW));
        }
        // per-channel vectors (a NULL scale is 1, a NULL bias 0)
        for (int i = tid; i < 4 * C; i += NT) {
            const int v = i / C, c = i - v * C;
            const float *src = v == 0 ? a.s0 : v == 1 ? a.b0 : v == 2 ? a.s2 : a.b2;
            reinterpret_cast<float *>(smem + OFF_VEC)[i] = src ? src[c] : (v == 0 || v == 2 ? 1.0f : 0.0f);
        }
        const float *vec = reinterpret_cast<const float *>(smem + OFF_VEC);
        u32x4 cst[CPT];
        chunk_load(a, 0, tid, cst);
        chunk_store(ring, tid, cst);
        // the first block's halo
        {
            const Blk k0 = decode(a, rstart * NW + wv);
            for (int s = 0; s < HSTEPS; s++) {
                u32x4 v[HSTEP];
                uint32_t d[HSTEP];
                halo_step_load(a, k0, s, lane, v, d);
                halo_step_store(reg, v, d);
            }
        }
        __syncthreads();

        // per-lane conv constants: A operand row (s, o) and tap row i = q - s
        const int cs = jl >> 3, co = jl & 7;
        const int ti = q - cs;
        const bool tap_ok = ti >= 0 && ti <= 2;
        const uint32_t a_off = (uint32_t)(tap_ok ? ti : 0) * GROW + (uint32_t)co * 16;
        // D rows of this lane: block row q >> 1, channels 8g + 4 (q & 1) + e
        const int drow = q >> 1, dch = 4 * (q & 1);

        int slot = 0;
        for (int r = 0; r < nr; r++) {
            const Blk k = decode(a, (rstart + r) * NW + wv);

            // 1. grouped conv, one group at a time.  Group g's d values overwrite
            //    only bytes of channels 8g..8g+7 of the wave's first 32 halo
            //    pixels, which later groups do not read, and this group's own
            //    halo reads precede the writes in the wave's LDS queue.
#pragma unroll
            for (int g = 0; g < NG; g++) {
                float4v acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int dj = 0; dj < 3; dj++) {
                    const u32x4 av = tap_ok ? lds16(gwl, a_off + (uint32_t)(dj * C + GW * g) * 16)
                                            : u32x4{0u, 0u, 0u, 0u};
                    const u32x4 bv = lds16(reg, (uint32_t)(q * HC + jl + dj) * PB + (uint32_t)g * 16);
                    acc = T::mfma(av, bv, acc);
                }
                const int c = GW * g + dch;
                const float4v sc = *reinterpret_cast<const float4v *>(vec + c);
                const float4v bi = *reinterpret_cast<const float4v *>(vec + C + c);
                float v[4];
#pragma unroll
                for (int e = 0; e < 4; e++)
                    v[e] = fmaf(acc[e], sc[e], bi[e]);
                *reinterpret_cast<u32x2 *>(reg + (uint32_t)(drow * BC + jl) * PB + (uint32_t)c * 2) =
                    u32x2{T::pack2(v[0], v[1]), T::pack2(v[2], v[3])};
            }
            // 2. d comes back as the expand's B fragments
            u32x4 dfr[2][KST];
#pragma unroll
            for (int nt = 0; nt < 2; nt++)
#pragma unroll
                for (int kk = 0; kk < KST; kk++)
                    dfr[nt][kk] = (32 * kk + 8 * q < C)
                                      ? lds16(reg, (uint32_t)(nt * BC + jl) * PB + (uint32_t)(32 * kk + 8 * q) * 2)
                                      : u32x4{0u, 0u, 0u, 0u};

            // 3. FFN over the hidden chunks; the next block's halo arrives meanwhile
            const bool more = r + 1 < nr;
            const Blk kn = decode(a, (rstart + r + 1) * NW + wv);
            float4v acc[2][MO];
#pragma unroll
            for (int nt = 0; nt < 2; nt++)
#pragma unroll
                for (int mo = 0; mo < MO; mo++)
                    acc[nt][mo] = float4v{0.f, 0.f, 0.f, 0.f};
            for (int ch = 0; ch < a.nch; ch++) {
                const int nxt = ch + 1 < a.nch ? ch + 1 : 0;
                chunk_load(a, nxt, tid, cst);
                u32x4 hv[HSTEP];
                uint32_t hd[HSTEP];
                const bool hstep = more && ch < HSTEPS;
                if (hstep)
                    halo_step_load(a, kn, ch, lane, hv, hd);

                const uint8_t *cur = ring + slot * CHB;
                float s1v[8], b1v[8];
                {
                    const float4v s_lo = *reinterpret_cast<const float4v *>(cur + W1B + W2B + 32 * q);
                    const float4v s_hi = *reinterpret_cast<const float4v *>(cur + W1B + W2B + 32 * q + 16);
                    const float4v b_lo = *reinterpret_cast<const float4v *>(cur + W1B + W2B + 128 + 32 * q);
                    const float4v b_hi = *reinterpret_cast<const float4v *>(cur + W1B + W2B + 128 + 32 * q + 16);
#pragma unroll
                    for (int e = 0; e < 4; e++) {
                        s1v[e] = s_lo[e];
                        s1v[4 + e] = s_hi[e];
                        b1v[e] = b_lo[e];
                        b1v[4 + e] = b_hi[e];
                    }
                }
                u32x4 a1[2][KST];
#pragma unroll
                for (int t = 0; t < 2; t++)
#pragma unroll
                    for (int kk = 0; kk < KST; kk++)
                        a1[t][kk] = lds16(cur, (uint32_t)(t * KST + kk) * 1024 + (uint32_t)lane * 16);
                u32x4 gfr[2];
#pragma unroll
                for (int nt = 0; nt < 2; nt++) {
                    float u[8];
#pragma unroll
                    for (int t = 0; t < 2; t++) {
                        float4v e = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                        for (int kk = 0; kk < KST; kk++)
                            e = T::mfma(a1[t][kk], dfr[nt][kk], e);
#pragma unroll
                        for (int i = 0; i < 4; i++)
                            u[4 * t + i] = act(fmaf(e[i], s1v[4 * t + i], b1v[4 * t + i]));
                    }
                    gfr[nt] = u32x4{T::pack2(u[0], u[1]), T::pack2(u[2], u[3]), T::pack2(u[4], u[5]),
                                    T::pack2(u[6], u[7])};
                }
#pragma unroll
                for (int mo = 0; mo < MO; mo++) {
                    const u32x4 a2 = lds16(cur, (uint32_t)W1B + (uint32_t)mo * 1024 + (uint32_t)lane * 16);
#pragma unroll
                    for (int nt = 0; nt < 2; nt++)
                        acc[nt][mo] = T::mfma(a2, gfr[nt], acc[nt][mo]);
                }
                chunk_store(ring + (slot ^ 1) * CHB, tid, cst);
                if (hstep)
                    halo_step_store(reg, hv, hd);
                __syncthreads();
                slot ^= 1;
            }
            // halo steps the chunks did not cover
            if (more) {
                for (int s = a.nch; s < HSTEPS; s++) {
                    u32x4 hv[HSTEP];
                    uint32_t hd[HSTEP];
                    halo_step_load(a, kn, s, lane, hv, hd);
                    halo_step_store(reg, hv, hd);
                }
            }

            // 4. epilogue: y = x + s2 * acc + b2 for the block's valid pixels
            if (k.valid) {
#pragma unroll
                for (int nt = 0; nt < 2; nt++) {
                    const int h = k.r0 + nt, w = k.c0 + jl;
                    if (h >= a.H || w >= a.W)
                        continue;
                    const size_t pix = ((size_t)k.n * a.H + h) * a.W + w;
#pragma unroll
                    for (int mo = 0; mo < MO; mo++) {
                        const int c = 16 * mo + 4 * q;
                        const u32x2 xv = *reinterpret_cast<const u32x2 *>(a.x + pix * C + c);
                        const float4v sc = *reinterpret_cast<const float4v *>(vec + 2 * C + c);
                        const float4v bi = *reinterpret_cast<const float4v *>(vec + 3 * C + c);
                        float o[4];
#pragma unroll
                        for (int e = 0; e < 4; e++)
                            o[e] = fmaf(acc[nt][mo][e], sc[e], bi[e]);
                        const u32x2 ov = {T::pack2(T::lo(xv[0]) + o[0], T::hi(xv[0]) + o[1]),
                                          T::pack2(T::lo(xv[1]) + o[2], T::hi(xv[1]) + o[3])};
                        *reinterpret_cast<u32x2 *>(a.y + pix * C + c) = ov;
                    }
                }
            }
        }
    }
};

template <int C, int NW, typename T, int ACT>
__global__ __launch_bounds__(NW * 64, 1) void gblock_kernel(Args a) {
    extern __shared__ __attribute__((aligned(256))) uint8_t smem[];
    GB<C, NW, T, ACT>::run(a, smem);
}

// waves per workgroup for a channel count: 8 where their halo regions fit
constexpr int nw_for(int C) { return C <= 96 ? 8 : 4; }

template <int C>
constexpr size_t lds_for() { return (size_t)GB<C, nw_for(C), F16, ACT_RELU>::LDS; }

template <int C>
hipError_t launch_c(const void *x, void *y, const GBlockW &w, const Shape &s, hipStream_t st) {
    constexpr int NW = nw_for(C);
    Args a{};
    a.x = (const uint16_t *)x;
    a.y = (uint16_t *)y;
    a.gw = (const uint16_t *)w.gw;
    a.s0 = w.s0;
    a.b0 = w.b0;
    a.w1 = (const uint16_t *)w.w1;
    a.s1 = w.s1;
    a.b1 = w.b1;
    a.w2 = (const uint16_t *)w.w2;
    a.s2 = w.s2;
    a.b2 = w.b2;
    a.H = s.H;
    a.W = s.W;
    a.EC = s.E * C;
    a.nch = (a.EC + 31) / 32;
    a.RP = (s.H + 1) / 2;
    a.SEG = (s.W + 15) / 16;
    const int64_t nb = (int64_t)s.N * a.RP * a.SEG;
    if (nb > ((int64_t)1 << 30))
        return hipErrorInvalidValue;
    a.nblocks = (int)nb;
    const int rounds = (int)((nb + NW - 1) / NW);
    const int cus = device_cu_count();
    const int G = rounds < cus ? rounds : cus;
    a.rbase = rounds / G;
    a.rextra = rounds % G;
    a.xcd_map = (G % 8 == 0) ? 1 : 0;
    const size_t lds = GB<C, NW, F16, ACT_RELU>::LDS;
    hipError_t e;
#define CF_GB_LAUNCH(TT, AC)                                           \
    {                                                                  \
        auto kf = gblock_kernel<C, NW, TT, AC>;                        \
        if ((e = allow_full_lds((const void *)kf)) != hipSuccess)      \
            return e;                                                  \
        hipLaunchKernelGGL(kf, dim3(G), dim3(NW * 64), lds, st, a);    \
    }
    if (s.bf16) {
        switch (s.act) {
        case ACT_GELU: CF_GB_LAUNCH(BF16, ACT_GELU) break;
        case ACT_RELU: CF_GB_LAUNCH(BF16, ACT_RELU) break;
        default: CF_GB_LAUNCH(BF16, ACT_NONE) break;
        }
    } else {
        switch (s.act) {
        case ACT_GELU: CF_GB_LAUNCH(F16, ACT_GELU) break;
        case ACT_RELU: CF_GB_LAUNCH(F16, ACT_RELU) break;
        default: CF_GB_LAUNCH(F16, ACT_NONE) break;
        }
    }
#undef CF_GB_LAUNCH
    return hipGetLastError();
}

}  // namespace gblk
}  // namespace cf
