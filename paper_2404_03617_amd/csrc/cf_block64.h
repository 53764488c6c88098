// cf_block64.h -- fused ConvFirst block for C = 64 channels, fp16 I/O, on
// gfx950.  Instantiated per depth-wise size in cf_block64_k*.hip.
//
// The block (Sec. 5.3 of Lavin, arXiv:2404.03617, norms folded to scale and
// bias) is evaluated by one persistent workgroup of 8 waves per CU with the
// block-fusion schedule of Sec. 5.3.1 / 5.5.1.  Differences from the generic
// kernel in cf_fused_impl.h, all aimed at the VALU and LDS budgets of the
// C = 64 case:
//
//  * Work is dealt in blocks of 32 consecutive pixels (N*H*W flattened).  Each
//    workgroup owns a contiguous range of blocks (ranges of neighbouring
//    workgroups sit on the same XCD, so halo rows shared by two ranges hit the
//    same L2) and walks it in tiles of up to 12 blocks.  In a 12-block tile
//    waves 0-3 take two blocks (64 pixels) and waves 4-7 one block; waves w
//    and w+4 share a SIMD, so every SIMD carries three blocks.
//  * W1, W2 (with s1, s2 folded in) and b1 stay in LDS for the whole kernel.
//  * The input tile plus halo is copied into LDS by LDS-DMA (global_load_lds,
//    1 KB per wave instruction, no registers); the copies of the next tile
//    are issued when the FFN of the current one starts and land while it
//    runs.  Pixels sit 144 bytes apart (128 data + 16 pad): eight
//    lanes reading the same channel chunk of eight neighbouring pixels hit
//    eight different bank groups, and every tap is the pixel's base address
//    plus a compile-time offset (fixed row stride), so the depth-wise loop
//    issues no address arithmetic.  Taps that fall outside the pixel's image
//    are redirected, row by row, to a zero area.
//  * Depth-wise conv on the VALU in packed fp16.  A two-block wave lets each
//    lane compute one pixel for all 16 channels of a K step; the taps are then
//    wave-uniform (broadcast LDS reads), and one v_permlane32_swap per
//    register pair rearranges the result into the two MFMA B fragments.  A
//    one-block wave uses the B-fragment lane layout directly.
//  * FFN per 32-hidden chunk on v_mfma_f32_32x32x16_f16 with swapped operands
//    (weights = A, pixels = B), the sigma/tau row orders of cf_fused_impl.h,
//    b1 as a fifth expand K step (a b1/4 fragment against a constant-one B
//    fragment), GELU evaluated on interleaved fp16 pairs.
//  * Accumulators start at x/4 + b2/4 read from the LDS halo (residual), the
//    activation variable is u/4 (exact power-of-two scaling), output 4*acc.
#pragma once
#include "cf_fused_impl.h"

namespace cf {
namespace b64 {

using fused::FastDiv;
using fused::fdiv;
using fused::mfma32;
using fused::float16v;
using fused::sigma_row;
using fused::tau_row;

constexpr int C = 64;
constexpr int NWAVE = 8;
constexpr int NT = NWAVE * 64;
constexpr int KST = C / 16;          // expand K steps
constexpr int CB = C / 32;           // 32-channel output blocks
constexpr int MAX_TB = 16;           // blocks per tile (two per wave at most)
constexpr int PIX = 144;             // LDS bytes per halo pixel
constexpr int CHUNK_W1 = (KST + 1) * 1024;  // W1 fragments of one 32-hidden chunk, then the b1 fragment
constexpr int CHUNK_W2 = 2 * CB * 1024;
constexpr float QS = 0.25f;

struct Args {
    const uint16_t *x;
    uint16_t *y;
    const uint16_t *dw_w;
    const float *s0, *b0;
    const uint16_t *w1;
    const float *s1, *b1;
    const uint16_t *w2;
    const float *s2, *b2;
    int H, W, NH;        // NH = N*H (global image rows)
    int nch;             // hidden chunks = E*C/32
    uint32_t P;          // N*H*W < 2^31
    FastDiv divW, divH;
    int nblocks;         // ceil(P / 32)
    int range_base, range_extra;  // blocks per workgroup: base (+1 for the first `extra`)
    int tile_max;        // largest tile, <= MAX_TB blocks
    uint32_t rs;         // LDS bytes per halo row: (W + 2*pad) * PIX
    int halo_rows;       // data rows of the halo buffer
    // LDS byte offsets
    uint32_t off_w2, off_b1, off_cst, off_dwt, off_halo, off_zero, off_trash;
};

// LDS map: [W1 + b1 nch*5 KB][W2 nch*4 KB][cst 512 B][taps k*k*128 B]
//          [halo halo_rows * rs][zero area][trash 1 KB]
struct Layout {
    uint32_t w2, b1, cst, dwt, halo, zero, trash, total;
};

inline Layout layout_for(int nch, int k, int halo_rows, uint32_t rs) {
    Layout L;
    L.w2 = (uint32_t)nch * CHUNK_W1;
    L.b1 = 0;  // the b1 fragments sit in the W1 chunks
    L.cst = L.w2 + (uint32_t)nch * CHUNK_W2;
    L.dwt = L.cst + 512;
    L.halo = (L.dwt + (uint32_t)k * k * 128 + 255) & ~255u;
    L.zero = L.halo + (uint32_t)halo_rows * rs;
    L.trash = (L.zero + (uint32_t)k * PIX + 128 + 15) & ~15u;
    L.total = L.trash + 1024;
    return L;
}

// halo rows a tile of tb blocks can touch (data rows, without the zero area)
inline int halo_rows_for(int tb, int k, int W, int64_t NH) {
    int64_t span = (int64_t)(32 * tb - 1) / W + 2;
    if (span > NH)
        span = NH;
    return (int)span + 2 * (k / 2);
}

__device__ __forceinline__ uint32_t lds_addr(const uint8_t *p) {
    return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const uint8_t *)p;
}
__device__ __forceinline__ u32x4 ld16(const uint8_t *base, uint32_t off) {
    return *reinterpret_cast<const u32x4 *>(base + off);
}
__device__ __forceinline__ half2v h2(uint32_t w) { return __builtin_bit_cast(half2v, w); }
__device__ __forceinline__ uint32_t u32(half2v v) { return __builtin_bit_cast(uint32_t, v); }

template <int KS, int ACT>
struct K64 {
    static constexpr int PAD = KS / 2;

    // ---- activation of 2*NP fp32 values (scaled by 1/4) into NP packed pairs.
    // Written stage by stage so the NP dependency chains interleave.
    template <int NP>
    static __device__ __forceinline__ void activate(const float *a, uint32_t *out) {
        half2v w[NP];
#pragma unroll
        for (int p = 0; p < NP; p++) {
            w[p].x = (_Float16)a[2 * p];
            w[p].y = (_Float16)a[2 * p + 1];
        }
        if constexpr (ACT == ACT_GELU) {
            half2v s[NP], q[NP];
#pragma unroll
            for (int p = 0; p < NP; p++)
                s[p] = w[p] * w[p];
#pragma unroll
            for (int p = 0; p < NP; p++)
                q[p] = __builtin_elementwise_fma(s[p], splat2(GELU_Q4), splat2(GELU_Q3));
#pragma unroll
            for (int p = 0; p < NP; p++)
                q[p] = __builtin_elementwise_fma(s[p], q[p], splat2(GELU_Q2));
#pragma unroll
            for (int p = 0; p < NP; p++)
                q[p] = __builtin_elementwise_fma(s[p], q[p], splat2(GELU_Q1));
#pragma unroll
            for (int p = 0; p < NP; p++)
                q[p] = __builtin_elementwise_fma(s[p], q[p], splat2(GELU_Q0));
#pragma unroll
            for (int p = 0; p < NP; p++)
                q[p] = __builtin_elementwise_min(
                    __builtin_elementwise_max(__builtin_elementwise_fma(w[p], q[p], splat2(0.5f)), splat2(0.0f)),
                    splat2(1.0f));
#pragma unroll
            for (int p = 0; p < NP; p++)
                out[p] = u32(w[p] * q[p]);
        } else if constexpr (ACT == ACT_RELU) {
#pragma unroll
            for (int p = 0; p < NP; p++)
                out[p] = u32(__builtin_elementwise_max(w[p], splat2(0.0f)));
        } else {
#pragma unroll
            for (int p = 0; p < NP; p++)
                out[p] = u32(w[p]);
        }
    }

    // ---- one-time staging: weights in MFMA fragment order with s1/s2 folded,
    // b1/4 in expand register order, per-channel constants, depth-wise taps.
    static __device__ void stage(const Args &a, uint8_t *smem, int tid) {
        const int pieces = a.nch * 512;  // 16-byte pieces: 256 of W1 + 256 of W2 per chunk
        for (int p = tid; p < pieces; p += NT) {
            const int ch = p >> 9, r = p & 511;
            const int lane = r & 63, f = r >> 6;  // f < 4: W1 K step; f >= 4: W2 (cb, kk)
            const int hh = lane >> 5, mm = lane & 31;
            const uint16_t *src;
            float sc;
            uint32_t dst;
            if (f < KST) {
                const int row = ch * 32 + sigma_row(mm);
                src = a.w1 + (size_t)row * C + f * 16 + 8 * hh;
                sc = a.s1 ? a.s1[row] : 1.0f;
                dst = (uint32_t)ch * CHUNK_W1 + (uint32_t)(f * 64 + lane) * 16;
            } else {
                const int g = f - KST, cb = g >> 1, kk = g & 1;
                const int row = cb * 32 + tau_row(mm);
                src = a.w2 + (size_t)row * (a.nch * 32) + ch * 32 + 16 * kk + 8 * hh;
                sc = a.s2 ? a.s2[row] : 1.0f;
                dst = a.off_w2 + (uint32_t)ch * CHUNK_W2 + (uint32_t)(g * 64 + lane) * 16;
            }
            Pack8 v;
            v.u = *reinterpret_cast<const u32x4 *>(src);
            if (sc != 1.0f) {
#pragma unroll
                for (int q = 0; q < 4; q++)
                    v.w[q] = F16::pack2(F16::lo(v.w[q]) * sc, F16::hi(v.w[q]) * sc);
            }
            *reinterpret_cast<u32x4 *>(smem + dst) = v.u;
        }
        // b1 / 4 as the A fragment of a fifth expand K step: row m of chunk ch
        // (hidden ch*32 + sigma(m)) holds b1/4 at k = 0 and zeros elsewhere; it
        // meets a constant B fragment that is 1 at k = 0 for every pixel.
        for (int p = tid; p < a.nch * 64; p += NT) {
            const int ch = p >> 6, lane = p & 63;
            u32x4 v = {0u, 0u, 0u, 0u};
            if (lane < 32 && a.b1) {
                const _Float16 bv = (_Float16)(a.b1[ch * 32 + sigma_row(lane)] * QS);
                v[0] = (uint32_t)__builtin_bit_cast(uint16_t, bv);
            }
            *reinterpret_cast<u32x4 *>(smem + (uint32_t)ch * CHUNK_W1 + (uint32_t)(KST * 64 + lane) * 16) = v;
        }
        for (int c = tid; c < C; c += NT) {
            reinterpret_cast<_Float16 *>(smem + a.off_cst)[c] = (_Float16)((a.s0 ? a.s0[c] : 1.0f) * QS);
            reinterpret_cast<_Float16 *>(smem + a.off_cst + 128)[c] = (_Float16)((a.b0 ? a.b0[c] : 0.0f) * QS);
            reinterpret_cast<float *>(smem + a.off_cst + 256)[c] = a.b2 ? a.b2[c] * QS : 0.0f;
        }
        for (int p = tid; p < KS * KS * 8; p += NT)
            reinterpret_cast<u32x4 *>(smem + a.off_dwt)[p] = reinterpret_cast<const u32x4 *>(a.dw_w)[p];
    }

    // ---- halo copy of the tile starting at block t0 with nblk blocks.
    // Row r of the buffer holds global image row g_lo - PAD + r; pixel column c
    // (c = image column + PAD) starts at r*rs + c*PIX; 16-byte slot s of a row
    // interior belongs to pixel s / 9, chunk s % 9 (chunk 8 is padding and gets
    // a copy of chunk 7).
    static __device__ __forceinline__ void tile_rows(const Args &a, int t0, int nblk, uint32_t &g_lo, int &rows) {
        const uint32_t p0 = (uint32_t)t0 * 32;
        uint32_t pend = p0 + (uint32_t)nblk * 32;
        if (pend > a.P)
            pend = a.P;
        g_lo = fdiv(p0, a.divW);
        rows = (int)(fdiv(pend - 1, a.divW) - g_lo) + 1 + 2 * PAD;
    }

    // ---- halo copy through LDS-DMA.  Row r of the buffer holds global image
    // row g_lo - PAD + r; pixel column c (= image column + PAD) starts at
    // r*rs + c*PIX.  The interior of a buffer row (W pixels from column PAD)
    // is 9W consecutive 16-byte slots: slot s belongs to pixel s / 9, chunk
    // s % 9, where chunk 8 is padding that receives a second copy of chunk 7
    // and is never read.  One DMA instruction fills 64 consecutive slots
    // (1 KB): wave wv fills slots 64 wv .. 64 wv + 63 of every row (9W <= 512),
    // with the lanes past the last slot switched off so that the pad columns
    // keep their zeros.  Rows outside the images are not copied (no tap reads
    // them).  The lane mask goes into EXEC inside the copy's instruction
    // group.
    struct HaloLane {
        uint32_t goff;  // byte offset in the image row of this lane's slot
        uint32_t loff;  // LDS byte offset of this wave's part inside a buffer row
        uint64_t mask;  // lanes whose slot lies inside the row
    };
    static __device__ __forceinline__ HaloLane halo_lane(const Args &a, int wv, int lane) {
        HaloLane hl;
        const int s0 = 64 * __builtin_amdgcn_readfirstlane(wv), sl = s0 + lane, px = sl / 9, q = sl % 9;
        hl.goff = (uint32_t)px * (C * 2) + (uint32_t)(q < 8 ? q : 7) * 16;
        hl.loff = (uint32_t)PAD * PIX + (uint32_t)s0 * 16;
        hl.mask = __ballot(sl < 9 * a.W);
        return hl;
    }
    // The next tile's copy, set up once per tile: buffer row r holds image row
    // (over N*H) g_lo - PAD + r, and rows rlo .. rlo + span - 1 are the ones
    // inside the images (span = 0 for a wave whose lanes all lie past the
    // row's end, or when there is no next tile).  gbase is the global address
    // of row rlo -- always a valid image row, so a copy that is not needed can
    // read it harmlessly.
    struct NextHalo {
        const uint8_t *gbase;
        uint32_t rlo, span;
    };
    static __device__ __forceinline__ NextHalo next_halo(const Args &a, const HaloLane &hl, uint32_t g_lo,
                                                         int rows) {
        int rlo = PAD - (int)g_lo;
        if (rlo < 0)
            rlo = 0;
        int rhi = a.NH - (int)g_lo + PAD;
        if (rhi > rows)
            rhi = rows;
        if (hl.mask == 0 || rhi < rlo)
            rhi = rlo;
        NextHalo nh;
        nh.rlo = (uint32_t)rlo;
        nh.span = (uint32_t)(rhi - rlo);
        nh.gbase = reinterpret_cast<const uint8_t *>(a.x) +
                   (size_t)((int)g_lo - PAD + rlo) * (size_t)((uint32_t)a.W * (C * 2));
        return nh;
    }
    // Copy buffer row r.  Branch-free, so that an FFN step stays one basic
    // block: for a row that is not needed every lane reads the first 16 bytes
    // of row rlo into a trash area instead (the mask never goes empty).
    static __device__ __forceinline__ void issue_row(const Args &a, uint32_t lds_base, const HaloLane &hl,
                                                     const NextHalo &nh, int r) {
        // okm = all ones when rlo <= r < rlo + span; masks rather than
        // selects, which the compiler would turn back into a branch
        const int d = r - (int)nh.rlo;
        const uint32_t okm = (uint32_t)(~(d >> 31) & ((d - (int)nh.span) >> 31));
        const uint64_t okm64 = (uint64_t)(int64_t)(int32_t)okm;
        const uint32_t row_off = ((uint32_t)d & okm) * ((uint32_t)a.W * (C * 2));  // < 2^32: a few image rows
        const uint32_t dst = a.off_halo + (uint32_t)r * a.rs + hl.loff;
        const uint32_t lds = lds_base + a.off_trash + ((dst - a.off_trash) & okm);
        fused::dma16m_at(nh.gbase + row_off, hl.goff & okm, lds, hl.mask | ~okm64);
    }
    static __device__ __forceinline__ void issue_halo(const Args &a, uint32_t lds_base, const HaloLane &hl,
                                                      const NextHalo &nh, int rows) {
        for (int r = 0; r < rows; r++)
            issue_row(a, lds_base, hl, nh, r);
    }

    // Base addresses of the KS tap rows of a pixel: the top-left tap of the
    // pixel's window plus i*rs for row i, or (for rows outside the pixel's
    // image, and for invalid pixels) an address that lands every tap of that
    // row in the zero area.
    static __device__ __forceinline__ void tap_bases(const Args &a, uint32_t pix, bool valid, uint32_t g_lo,
                                                     uint32_t extra, uint32_t (&base)[KS], uint32_t &centre) {
        uint32_t topleft = 0, hh = 0;
        if (valid) {
            const uint32_t gg = fdiv(pix, a.divW);
            const uint32_t wc = pix - gg * (uint32_t)a.W;
            hh = gg - fdiv(gg, a.divH) * (uint32_t)a.H;
            topleft = a.off_halo + (gg - g_lo) * a.rs + wc * PIX;
        }
        centre = topleft + PAD * a.rs + PAD * PIX + extra;
#pragma unroll
        for (int i = 0; i < KS; i++) {
            const int hr = (int)hh + i - PAD;
            const bool in = valid && hr >= 0 && hr < a.H;
            base[i] = (in ? topleft + (uint32_t)i * a.rs : a.off_zero) + extra;
        }
    }

    // ---- depth-wise conv (Sec. 4.1.1, degenerate group width 1) of NQ 16-byte
    // channel chunks.  Chunk qi of a lane reads pixel data at
    // base[i] + j*PIX + qi*vstep and taps at wbase + (i*KS + j)*128 + qi*wstep
    // (taps are read from LDS: a scalar load would share the lgkm counter with
    // the LDS reads and force a full drain before every use).  The work is cut
    // into units of one tap row of one chunk; the reads of unit u + DIST are
    // issued before unit u is computed, through a register ring.
    static constexpr int DIST = KS <= 1 ? 6 : KS <= 3 ? 3 : 1;
    template <int NQ>
    static __device__ __forceinline__ void dw_conv(const uint8_t *smem, const uint32_t (&base)[KS], uint32_t wbase,
                                                   uint32_t vstep, uint32_t wstep, uint32_t cst, uint32_t cstep,
                                                   uint32_t (&d)[NQ][4]) {
        constexpr int NU = NQ * KS, R = DIST + 1;
        u32x4 vb[R][KS], wb[R][KS];
#pragma unroll
        for (int u = 0; u < DIST && u < NU; u++) {
            const int qi = u / KS, i = u % KS;
#pragma unroll
            for (int j = 0; j < KS; j++) {
                vb[u % R][j] = ld16(smem, base[i] + (uint32_t)(j * PIX + qi * vstep));
                wb[u % R][j] = ld16(smem, wbase + (uint32_t)((i * KS + j) * 128 + qi * wstep));
            }
        }
        half2v acc[4];
#pragma unroll
        for (int u = 0; u < NU; u++) {
            const int qi = u / KS, i = u % KS;
            if (u + DIST < NU) {
                const int un = u + DIST, qn = un / KS, in = un % KS;
#pragma unroll
                for (int j = 0; j < KS; j++) {
                    vb[un % R][j] = ld16(smem, base[in] + (uint32_t)(j * PIX + qn * vstep));
                    wb[un % R][j] = ld16(smem, wbase + (uint32_t)((in * KS + j) * 128 + qn * wstep));
                }
            }
            if (i == 0) {
#pragma unroll
                for (int e = 0; e < 4; e++)
                    acc[e] = splat2(0.0f);
            }
#pragma unroll
            for (int j = 0; j < KS; j++) {
                Pack8 v, w;
                v.u = vb[u % R][j];
                w.u = wb[u % R][j];
#pragma unroll
                for (int e = 0; e < 4; e++)
                    acc[e] = __builtin_elementwise_fma(h2(v.w[e]), h2(w.w[e]), acc[e]);
            }
            if (i == KS - 1) {
                Pack8 sp, bp;
                sp.u = ld16(smem, cst + (uint32_t)(qi * cstep));
                bp.u = ld16(smem, cst + 128 + (uint32_t)(qi * cstep));
#pragma unroll
                for (int e = 0; e < 4; e++)
                    d[qi][e] = u32(__builtin_elementwise_fma(acc[e], h2(sp.w[e]), h2(bp.w[e])));
            }
            // this unit: the reads of unit u + DIST, then its FMAs (pinned for
            // small kernels; for k >= 5 the order is left to the compiler,
            // whose group solver does not finish on that many units)
            if constexpr (KS <= 3) {
                __builtin_amdgcn_sched_group_barrier(0x100, 2 * KS, 0);
                __builtin_amdgcn_sched_group_barrier(0x002, 4 * KS, 0);
            }
        }
    }

    // two-block wave: lane l computes pixel l of the wave's 64 (block j0 for
    // l < 32, block j1 above) for all 16 channels of each K step (taps are the
    // same for every lane), then swaps halves into the two B fragments.
    static __device__ __forceinline__ void dw_pair(const Args &a, const uint8_t *smem, const uint32_t (&base)[KS],
                                                   u32x4 (&dfr)[KST][2]) {
        uint32_t d[2 * KST][4];
        dw_conv<2 * KST>(smem, base, a.off_dwt, 16u, 16u, a.off_cst, 16u, d);
        // lanes 32-63 of chunk 2ks <-> lanes 0-31 of chunk 2ks+1
#pragma unroll
        for (int ks = 0; ks < KST; ks++)
#pragma unroll
            for (int e = 0; e < 4; e++) {
                const auto r = __builtin_amdgcn_permlane32_swap(d[2 * ks][e], d[2 * ks + 1][e], false, false);
                dfr[ks][0][e] = r[0];
                dfr[ks][1][e] = r[1];
            }
    }

    // one-block wave: lane (h, m) computes channels 16ks + 8h .. +7 of pixel m
    // (the B-fragment layout; base already includes the 16h byte offset).
    static __device__ __forceinline__ void dw_single(const Args &a, const uint8_t *smem, const uint32_t (&base)[KS],
                                                     int h, u32x4 (&dfr)[KST][2]) {
        uint32_t d[KST][4];
        dw_conv<KST>(smem, base, a.off_dwt + (uint32_t)h * 16, 32u, 32u, a.off_cst + (uint32_t)h * 16, 32u, d);
#pragma unroll
        for (int ks = 0; ks < KST; ks++)
#pragma unroll
            for (int e = 0; e < 4; e++)
                dfr[ks][0][e] = d[ks][e];
    }

    // ---- residual start: acc = x/4 + b2/4 from the halo centre, MFMA layout
    // (lane (h, m): channels cb*32 + 16h .. +15 of pixel m of block b).
    template <int NB>
    static __device__ __forceinline__ void residual(const Args &a, const uint8_t *smem, const uint32_t (&centre)[2],
                                                    int h, float16v (&acc)[CB][2]) {
#pragma unroll
        for (int cb = 0; cb < CB; cb++) {
            const float16v bias = *reinterpret_cast<const float16v *>(smem + a.off_cst + 256 + (cb * 32 + 16 * h) * 4);
#pragma unroll
            for (int b = 0; b < NB; b++) {
                Pack8 v0, v1;
                v0.u = ld16(smem, centre[b] + (uint32_t)(cb * 64));
                v1.u = ld16(smem, centre[b] + (uint32_t)(cb * 64 + 16));
                float16v t;
#pragma unroll
                for (int q = 0; q < 4; q++) {
                    t[2 * q] = fmaf(F16::lo(v0.w[q]), QS, bias[2 * q]);
                    t[2 * q + 1] = fmaf(F16::hi(v0.w[q]), QS, bias[2 * q + 1]);
                    t[8 + 2 * q] = fmaf(F16::lo(v1.w[q]), QS, bias[8 + 2 * q]);
                    t[8 + 2 * q + 1] = fmaf(F16::hi(v1.w[q]), QS, bias[8 + 2 * q + 1]);
                }
                acc[cb][b] = t;
            }
        }
    }

    // ---- FFN over all hidden chunks (eq. e:ffn-eff): expand, phi, project.
    // Three-stage software pipeline over the chunks: step s issues the expand
    // MFMAs of chunk s, activates chunk s-1 (VALU) and issues the project
    // MFMAs of chunk s-2.  The three are independent, so the matrix and vector
    // instructions of a step are interleaved (one MFMA, then a run of VALU
    // instructions that execute while it runs) and no instruction waits on an
    // MFMA result issued in the same step.  Two expand accumulator sets (u0,
    // u1) and two activated sets (g0, g1) alternate between even and odd steps.
    template <int NB>
    static __device__ __forceinline__ void act_blocks(const float16v (&u)[2], uint32_t (&g)[16]) {
#pragma unroll
        for (int b = 0; b < NB; b++)
#pragma unroll
            for (int p0 = 0; p0 < 8; p0 += 4) {
                float v[8];
#pragma unroll
                for (int i = 0; i < 8; i++)
                    v[i] = u[b][2 * p0 + i];
                activate<4>(v, &g[b * 8 + p0]);
            }
    }

    struct Ffn {
        const uint8_t *w1p, *w2p;
        u32x4 ones;  // B fragment: 1 at k = 0 for every pixel (bias K step)
        uint32_t lds_base;  // LDS byte address of the dynamic area
        HaloLane hl;
        NextHalo nh;
    };

    template <int NB, bool EXP, bool ACTV, bool PROJ>
    static __device__ __forceinline__ void step(const Args &a, const Ffn &f, int s, const u32x4 (&dfr)[KST][2],
                                                float16v (&ue)[2], const float16v (&ua)[2], uint32_t (&ga)[16],
                                                const uint32_t (&gp)[16], float16v (&acc)[CB][2]) {
        // halo row s of the next tile (the tile touches at most nch + 2 rows)
        issue_row(a, f.lds_base, f.hl, f.nh, s);
        if constexpr (ACTV)
            act_blocks<NB>(ua, ga);
        if constexpr (EXP) {
            const uint8_t *wp = f.w1p + s * CHUNK_W1;
            const u32x4 bfr = *reinterpret_cast<const u32x4 *>(wp + KST * 1024);
#pragma unroll
            for (int b = 0; b < NB; b++)
                ue[b] = mfma32(bfr, f.ones, float16v{}, F16{});
#pragma unroll
            for (int ks = 0; ks < KST; ks++) {
                const u32x4 w1f = *reinterpret_cast<const u32x4 *>(wp + ks * 1024);
#pragma unroll
                for (int b = 0; b < NB; b++)
                    ue[b] = mfma32(w1f, dfr[ks][b], ue[b], F16{});
            }
        }
        if constexpr (PROJ) {
#pragma unroll
            for (int kk = 0; kk < 2; kk++)
#pragma unroll
                for (int cb = 0; cb < CB; cb++) {
                    const u32x4 w2f = *reinterpret_cast<const u32x4 *>(f.w2p + (s - 2) * CHUNK_W2 +
                                                                      (cb * 2 + kk) * 1024);
#pragma unroll
                    for (int b = 0; b < NB; b++) {
                        u32x4 hid;
#pragma unroll
                        for (int p = 0; p < 4; p++)
                            hid[p] = gp[b * 8 + kk * 4 + p];
                        acc[cb][b] = mfma32(w2f, hid, acc[cb][b], F16{});
                    }
                }
        }
        // Interleave: fragment reads ahead of their use, one MFMA, then the
        // VALU instructions that execute in its shadow.
        constexpr int NM = (EXP ? NB * (KST + 1) : 0) + (PROJ ? NB * 2 * CB : 0);
        constexpr int NV = ACTV ? NB * 64 : 0;
        if constexpr (NM > 0 && NV > 0) {
            constexpr int VPER = (NV - 8 + NM - 1) / NM;
            __builtin_amdgcn_sched_group_barrier(0x100, 3, 0);
            __builtin_amdgcn_sched_group_barrier(0x002, 8, 0);
#pragma unroll
            for (int i = 0; i < NM; i++) {
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x002, VPER, 0);
            }
        }
    }

    template <int NB>
    static __device__ __forceinline__ void ffn(const Args &a, uint8_t *smem, int lane, const HaloLane &hl,
                                               const NextHalo &nh, const u32x4 (&dfr)[KST][2],
                                               float16v (&acc)[CB][2]) {
        Ffn f;
        f.w1p = smem + lane * 16;
        f.w2p = smem + a.off_w2 + lane * 16;
        f.ones = u32x4{lane < 32 ? 0x3c00u : 0u, 0u, 0u, 0u};
        f.lds_base = lds_addr(smem);
        f.hl = hl;
        f.nh = nh;
        float16v u0[2], u1[2];
        uint32_t g0[16], g1[16];
        const int n = a.nch;  // even, >= 2
        step<NB, true, false, false>(a, f, 0, dfr, u0, u1, g1, g0, acc);
        step<NB, true, true, false>(a, f, 1, dfr, u1, u0, g0, g1, acc);
#pragma unroll 1
        for (int s = 2; s < n; s += 2) {
            step<NB, true, true, true>(a, f, s, dfr, u0, u1, g1, g0, acc);
            step<NB, true, true, true>(a, f, s + 1, dfr, u1, u0, g0, g1, acc);
        }
        step<NB, false, true, true>(a, f, n, dfr, u0, u1, g1, g0, acc);
        step<NB, false, false, true>(a, f, n + 1, dfr, u1, u0, g0, g1, acc);
    }

    template <int NB>
    static __device__ __forceinline__ int store(const Args &a, const uint32_t (&pix)[2], const bool (&valid)[2],
                                                int h, const float16v (&acc)[CB][2]) {
        int n = 0;
#pragma unroll
        for (int b = 0; b < NB; b++) {
            if (__builtin_amdgcn_read_exec() && __ballot(valid[b]))
                n += 2 * CB;
            if (!valid[b])
                continue;
#pragma unroll
            for (int cb = 0; cb < CB; cb++) {
                u32x4 o0, o1;
#pragma unroll
                for (int q = 0; q < 4; q++) {
                    o0[q] = F16::pack2(4.0f * acc[cb][b][2 * q], 4.0f * acc[cb][b][2 * q + 1]);
                    o1[q] = F16::pack2(4.0f * acc[cb][b][8 + 2 * q], 4.0f * acc[cb][b][8 + 2 * q + 1]);
                }
                u32x4 *dst = reinterpret_cast<u32x4 *>(a.y + (size_t)pix[b] * C + cb * 32 + 16 * h);
                dst[0] = o0;
                dst[1] = o1;
            }
        }
        return n;
    }

    static __device__ void run(const Args &a, uint8_t *smem) {
        const int tid = threadIdx.x;
        const int lane = tid & 63, wv = tid >> 6;
        const int h = lane >> 5, m = lane & 31;

        // block range of this workgroup; consecutive ranges on one XCD
        const int G = gridDim.x;
        const int g = (G % 8 == 0) ? (blockIdx.x % 8) * (G / 8) + blockIdx.x / 8 : blockIdx.x;
        const int lo = g * a.range_base + (g < a.range_extra ? g : a.range_extra);
        const int hi = lo + a.range_base + (g < a.range_extra ? 1 : 0);

        // zero the halo region and the zero area once; stage weights
        for (uint32_t i = a.off_halo / 16 + tid; i < (a.off_zero + KS * PIX + 128) / 16; i += NT)
            reinterpret_cast<u32x4 *>(smem)[i] = u32x4{0u, 0u, 0u, 0u};
        stage(a, smem, tid);
        __syncthreads();

        const HaloLane hl = halo_lane(a, wv, lane);
        // the range is cut into tiles of tile_max blocks and a last, smaller
        // one: a full tile gives every SIMD the same number of blocks
        const int range = hi - lo;
        const int nt = (range + a.tile_max - 1) / a.tile_max;
        if (nt > 0) {
            uint32_t g0;
            int r0;
            tile_rows(a, lo, range < a.tile_max ? range : a.tile_max, g0, r0);
            issue_halo(a, lds_addr(smem), hl, next_halo(a, hl, g0, r0), r0);
        }
        int pending = 0;  // output stores this wave issued after its last halo copies

        int t0 = lo;
        for (int it = 0; it < nt; it++) {
            const int nblk = (hi - t0) < a.tile_max ? (hi - t0) : a.tile_max;
            uint32_t g_lo;
            int rows;
            tile_rows(a, t0, nblk, g_lo, rows);
            (void)rows;
            // this wave's blocks: w (if w < nblk) and 8 + w (if 8 + w < nblk)
            const int nb = (wv < nblk ? 1 : 0) + (wv + 8 < nblk ? 1 : 0);
            const int jb[2] = {wv, wv + 8};

            // MFMA-layout pixels of lane (h, m) and their halo centres
            uint32_t pix[2], centre[2];
            bool valid[2];
#pragma unroll
            for (int b = 0; b < 2; b++) {
                pix[b] = (uint32_t)(t0 + jb[b]) * 32 + m;
                valid[b] = (b < nb) && pix[b] < a.P;
                uint32_t bs[KS];
                tap_bases(a, pix[b], valid[b], g_lo, (uint32_t)h * 32, bs, centre[b]);
            }

            // this wave's halo copies have landed (vector-memory operations
            // complete in order; the stores issued after them may still be
            // in flight) ...
            fused::wait_vmcnt_le(pending);
            __syncthreads();  // ... and every other wave's: the tile's halo is in LDS

            u32x4 dfr[KST][2];
            float16v acc[CB][2];
            if (nb == 2) {
                // depth-wise layout: lane l -> pixel l & 31 of block jb[l >> 5]
                const uint32_t pd = (uint32_t)(t0 + jb[h]) * 32 + m;
                uint32_t bs[KS], cdummy;
                tap_bases(a, pd, pd < a.P, g_lo, 0u, bs, cdummy);
                dw_pair(a, smem, bs, dfr);
                residual<2>(a, smem, centre, h, acc);
            } else if (nb == 1) {
                uint32_t bs[KS], cdummy;
                tap_bases(a, pix[0], valid[0], g_lo, (uint32_t)h * 16, bs, cdummy);
                dw_single(a, smem, bs, h, dfr);
                residual<1>(a, smem, centre, h, acc);
            }
            __syncthreads();  // the halo buffer is free
            // the next tile's halo streams into LDS, a row per FFN step
            const int t1 = t0 + nblk;
            uint32_t g1 = 0;
            int rows1 = 0;
            if (it + 1 < nt) {
                const int nblk1 = (hi - t1) < a.tile_max ? (hi - t1) : a.tile_max;
                tile_rows(a, t1, nblk1, g1, rows1);
            }
            const NextHalo nh = next_halo(a, hl, g1, rows1);
            pending = 0;
            if (nb == 2) {
                ffn<2>(a, smem, lane, hl, nh, dfr, acc);
                pending = store<2>(a, pix, valid, h, acc);
            } else if (nb == 1) {
                ffn<1>(a, smem, lane, hl, nh, dfr, acc);
                pending = store<1>(a, pix, valid, h, acc);
            } else {
                issue_halo(a, lds_addr(smem), hl, nh, rows1);
            }
            t0 = t1;
        }
        __builtin_amdgcn_s_waitcnt(0);
    }
};

template <int KS, int ACT>
__global__ __launch_bounds__(NT, 1) void block64_kernel(Args a) {
    extern __shared__ __attribute__((aligned(256))) uint8_t smem[];
    K64<KS, ACT>::run(a, smem);
}

// ---------------------------------------------------------------------------
// Host side.  Returns hipErrorInvalidConfiguration when the shape needs the
// generic kernel (W too wide for the fixed halo row, or LDS does not fit).
inline bool plan(int N, int H, int W, int E, int k, int max_range, int tb_limit, int &tb, int &halo_rows,
                 uint32_t &rs, Layout &L) {
    const int pad = k / 2;
    // a row of the halo is one DMA instruction per wave: 9W slots <= 8 * 64
    if (W > 56 || E * C % 32 != 0 || E * C / 32 > 8)
        return false;
    rs = (uint32_t)(W + 2 * pad) * PIX;
    const int64_t NH = (int64_t)N * H;
    const int nch = E * C / 32;
    // the next tile's halo rows are copied one per FFN step (nch + 2 steps),
    // so a tile may touch at most nch + 2 rows, unless every workgroup has a
    // single tile (the first tile is copied whole)
    for (tb = tb_limit < MAX_TB ? tb_limit : MAX_TB; tb >= 1; tb--) {
        halo_rows = halo_rows_for(tb, k, W, NH);
        L = layout_for(nch, k, halo_rows, rs);
        if (L.total <= 160 * 1024 && (halo_rows <= nch + 2 || max_range <= tb))
            return true;
    }
    return false;
}

template <int KS>
hipError_t launch_k(const void *x, void *y, const BlockW &w, const Shape &s, hipStream_t st) {
    const int64_t P = (int64_t)s.N * s.H * s.W;
    const int nblocks = (int)((P + 31) / 32);
    int G = device_cu_count();
    if (G > nblocks)
        G = nblocks;
    int tb, halo_rows;
    uint32_t rs;
    Layout L;
    int tb_limit = MAX_TB;
    if (s.cfg == CFG_HALF_TILE) {
        // half of the largest tile that fits
        int tb0, hr0;
        uint32_t rs0;
        Layout L0;
        if (!plan(s.N, s.H, s.W, s.E, KS, (nblocks + G - 1) / G, MAX_TB, tb0, hr0, rs0, L0))
            return hipErrorInvalidConfiguration;
        tb_limit = tb0 / 2 > 0 ? tb0 / 2 : 1;
    }
    if (!plan(s.N, s.H, s.W, s.E, KS, (nblocks + G - 1) / G, tb_limit, tb, halo_rows, rs, L))
        return hipErrorInvalidConfiguration;
    Args a{};
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
    a.H = s.H;
    a.W = s.W;
    a.NH = s.N * s.H;
    a.nch = s.E * C / 32;
    a.P = (uint32_t)P;
    a.divW = fused::make_fastdiv((uint32_t)s.W);
    a.divH = fused::make_fastdiv((uint32_t)s.H);
    a.nblocks = nblocks;
    a.range_base = a.nblocks / G;
    a.range_extra = a.nblocks % G;
    a.tile_max = tb;
    a.rs = rs;
    a.halo_rows = halo_rows;
    a.off_w2 = L.w2;
    a.off_b1 = L.b1;
    a.off_cst = L.cst;
    a.off_dwt = L.dwt;
    a.off_halo = L.halo;
    a.off_zero = L.zero;
    a.off_trash = L.trash;
    hipError_t e;
    switch (s.act) {
    case ACT_GELU: {
        auto kf = block64_kernel<KS, ACT_GELU>;
        if ((e = allow_full_lds((const void *)kf)))
            return e;
        hipLaunchKernelGGL(kf, dim3(G), dim3(NT), L.total, st, a);
        break;
    }
    case ACT_RELU: {
        auto kf = block64_kernel<KS, ACT_RELU>;
        if ((e = allow_full_lds((const void *)kf)))
            return e;
        hipLaunchKernelGGL(kf, dim3(G), dim3(NT), L.total, st, a);
        break;
    }
    default: {
        auto kf = block64_kernel<KS, ACT_NONE>;
        if ((e = allow_full_lds((const void *)kf)))
            return e;
        hipLaunchKernelGGL(kf, dim3(G), dim3(NT), L.total, st, a);
        break;
    }
    }
    return hipGetLastError();
}

}  // namespace b64

#define CF_B64_UNITS(X) X(1) X(3) X(5) X(7)
#define CF_DECL_B64(K) hipError_t launch_block64_k##K(const void *x, void *y, const BlockW &w, const Shape &s, hipStream_t st);
CF_B64_UNITS(CF_DECL_B64)

}  // namespace cf
