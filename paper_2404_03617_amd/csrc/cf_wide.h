// cf_wide.h -- fused ConvFirst block for C = 128 and C = 256 channels, fp16
// I/O, on gfx950.  Instantiated per channel count in cf_wide_c*.hip.
//
// Block fusion (Sec. 5.3.1 / 5.5.1 of Lavin, arXiv:2404.03617) with one
// persistent workgroup of 8 waves per CU.  A tile is 4 blocks of 32
// consecutive pixels (N*H*W flattened); block b belongs to the wave pair
// (b, b + 4), which shares a SIMD.  Each workgroup owns a contiguous range of
// blocks.
//
//  * Depth-wise conv in slabs of 128 channels, channel-major: lane l handles
//    channels 4*(l % 32) .. +3 of the slab with its taps held in registers;
//    each half-wave walks 8 pixels.  A tap is one 8-byte LDS read of the halo
//    (contiguous across the lanes) and two packed fp16 FMAs.  The result goes
//    through a small LDS buffer and is read back as MFMA B fragments, so no
//    weight is re-read per pixel.
//  * FFN (eq. e:ffn-eff) in steps of two 32-hidden chunks on
//    v_mfma_f32_32x32x16_f16 with swapped operands and the sigma/tau row
//    orders of cf_fused_impl.h.  In step s wave r of a pair expands chunk
//    2s + r (b1 through the C operand), applies phi on fp16 pairs and puts the
//    result in LDS; after a barrier each wave projects its half of the output
//    channels over both chunks.  The W1 fragments of a step and its W2
//    fragments live in two LDS buffers, each refilled by asynchronous
//    global->LDS copies while the other one is in use.  s1 scales the expand
//    accumulators, s2 the output.
//  * The halo region is reused for the weight buffers once the depth-wise conv
//    of a tile is done.
//  * Epilogue y = x + s2 Z + b2 with x read back from global memory (it was just
//    read for the halo) -- the residual costs no extra HBM traffic.
// The activation variable is scaled by 1/4 as in the other kernels.
#pragma once
#include "cf_fused_impl.h"

namespace cf {
namespace wide {

using fused::FastDiv;
using fused::fdiv;
using fused::float16v;
using fused::mfma32;
using fused::sigma_row;
using fused::tau_row;

// LDS byte address of a pointer into the dynamic LDS area
__device__ __forceinline__ uint32_t lds_addr(const uint8_t *p) {
    return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const uint8_t *)p;
}
// One LDS-DMA instruction (64 lanes x 16 bytes from base + voff to LDS
// address lds_addr .. + 1 KB), as fused::dma16s, with the destination given as
// an LDS address (no generic-pointer conversion in the callers' loops).
__device__ __forceinline__ void dma16s_at(const void *base, uint32_t voff, uint32_t lds_addr_) {
    const uint32_t lds = (uint32_t)__builtin_amdgcn_readfirstlane(lds_addr_);
    const uint64_t b = (uint64_t)(uintptr_t)base;
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)b);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(b >> 32));
    const uint64_t bu = ((uint64_t)hi << 32) | (uint64_t)lo;
    uint32_t saved;
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %3\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %1, %2\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved)
        : "v"(voff), "s"(bu), "s"(lds)
        : "memory");
}

constexpr int NW = 8;               // waves; two per 32-pixel block
constexpr int NBLK = 4;             // blocks per tile
constexpr int NT = NW * 64;
constexpr int CS = 128;              // channels per depth-wise slab
constexpr int HPX = CS * 2;          // halo bytes per pixel (one slab)
constexpr int DPX = CS * 2 + 16;     // D-buffer bytes per pixel (padded against bank conflicts)
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
    int H, W, NH;
    int nch;              // hidden chunks = E*C/32
    uint32_t P;
    FastDiv divW, divH;
    int range_base, range_extra;
    uint32_t rsl;         // halo row bytes: (W + 2*pad) * HPX
    uint32_t off_b1, off_s2b2, off_s1, off_g, off_d, off_big, off_zero;
};

template <int C>
struct Geo {
    static constexpr int KST = C / 16;
    static constexpr int CB = C / 32;
    static constexpr int NSLAB = C / CS;
    // weight buffers of a step (two chunks): LDS-DMA instructions of 1 KB at
    // a pitch of PITCH bytes
    static constexpr int PITCH = 1040;
    static constexpr int RPI = 1024 / (2 * C);      // W1 rows per instruction
    static constexpr int NIA = 64 / RPI;            // instructions of an A buffer (64 W1 rows)
    static constexpr int NIB = C / 8;               // instructions of a B buffer (C segments of 128 bytes)
    static constexpr int BUF_A = NIA * PITCH;
    static constexpr int BUF_B = NIB * PITCH;
};

struct Layout {
    uint32_t b1, s2b2, s1, g, d, big, zero, total;
};

// [b1/4 regs nch*128][4*s2 | b2  C*8][s1 regs nch*128][G 4 blocks x 2 chunks x 2 KB]
// [overlay: halo + D buffer  |  W1 buffers A0 A1 + W2 buffers B0 B1][zero]
template <int C>
inline Layout layout_for(int nch, int k, int halo_rows, uint32_t rsl) {
    Layout L;
    L.b1 = 0;
    L.s2b2 = L.b1 + (uint32_t)nch * 128;
    L.s1 = L.s2b2 + (uint32_t)C * 8;
    L.g = (L.s1 + (uint32_t)nch * 128 + 255) & ~255u;
    L.big = L.g + NBLK * 2 * 2048;
    const uint32_t halo = (uint32_t)halo_rows * rsl;
    L.d = L.big + ((halo + 255) & ~255u);
    const uint32_t hd = (L.d - L.big) + NBLK * 32 * DPX;
    const uint32_t bufs = 2 * (Geo<C>::BUF_A + Geo<C>::BUF_B);
    L.zero = L.big + (hd > bufs ? hd : bufs);
    L.total = L.zero + (uint32_t)k * HPX + 64;
    return L;
}

inline int halo_rows_for(int k, int W, int64_t NH) {
    int64_t span = (int64_t)(32 * NBLK - 1) / W + 2;
    if (span > NH)
        span = NH;
    return (int)span + 2 * (k / 2);
}

// Workgroup barrier that waits only for this wave's LDS traffic (lgkmcnt),
// not for its outstanding global->LDS copies: those are waited for
// explicitly, per buffer, with partial vmcnt waits.  The empty asm statements
// keep the compiler from moving memory accesses across the barrier.
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_s_waitcnt(0xC07F);  // vmcnt 63, expcnt 7, lgkmcnt 0
    __asm__ volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    __asm__ volatile("" ::: "memory");
}

__device__ __forceinline__ u32x4 ld16(const uint8_t *base, uint32_t off) {
    return *reinterpret_cast<const u32x4 *>(base + off);
}
__device__ __forceinline__ half2v h2(uint32_t w) { return __builtin_bit_cast(half2v, w); }
__device__ __forceinline__ uint32_t u32(half2v v) { return __builtin_bit_cast(uint32_t, v); }

template <int C, int KS, int ACT>
struct Kw {
    typedef Geo<C> G;
    static constexpr int KST = G::KST, CB = G::CB, NSLAB = G::NSLAB, PITCH = G::PITCH, RPI = G::RPI;
    static constexpr int CBH = CB / 2;  // output blocks per wave of a pair
    static constexpr int PAD = KS / 2;

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

    // ---- per-kernel staging of the small vectors (register order).
    // Expand register e = 4t + i of lane half h <-> hidden 16(t>>1) + 8h + 4(t&1) + i.
    template <int NTV = NT>
    static __device__ void stage_vectors(const Args &a, uint8_t *smem, int tid, int ch0 = 0, int nchv = -1) {
        if (nchv < 0)
            nchv = a.nch;
        for (int p = tid; p < nchv * 32; p += NTV) {
            const int ch = ch0 + (p >> 5), e = p & 31, hh = e >> 4, t = (e >> 2) & 3, i = e & 3;
            const int r = ch * 32 + 16 * (t >> 1) + 8 * hh + 4 * (t & 1) + i;
            reinterpret_cast<float *>(smem + a.off_b1)[p] = a.b1 ? a.b1[r] * QS : 0.0f;
            reinterpret_cast<float *>(smem + a.off_s1)[p] = a.s1 ? a.s1[r] : 1.0f;
        }
        for (int c = tid; c < C; c += NTV) {
            reinterpret_cast<float *>(smem + a.off_s2b2)[c] = 4.0f * (a.s2 ? a.s2[c] : 1.0f);
            reinterpret_cast<float *>(smem + a.off_s2b2 + 4 * C)[c] = a.b2 ? a.b2[c] : 0.0f;
        }

    }

    // ---- weight buffers.  Buffer A of step s holds the W1 fragments (rows in
    // sigma order) of chunks 2s and 2s + 1: fragment j*KST + ks; buffer B the
    // W2 fragments (rows in tau order): fragment j*2*CB + 2*cb + kk.
    // ---- weight buffers A0 A1 B0 B1 (step s uses A_(s&1) and B_(s&1)),
    // filled by LDS-DMA, wave wv issuing instructions wv, wv + NW, ...  Every LDS-DMA instruction reads contiguous runs of
    // memory (8 cache lines per KB, against 32 when a KB is gathered in
    // fragment order, which the vector memory unit serves about five times
    // slower), and the instructions sit PITCH bytes apart (16 of padding), so
    // that the fragment reads below hit 16 different bank groups per 16 lanes.
    //  * A (W1, 64 rows of C halves per step): row r of chunk j is numbered
    //    (q, u) with q = 2j + r / 16, u = r % 16, and sits in instruction
    //    u + 16 (q / RPI) at byte (q % RPI) * 2C.  The rows sigma(m) read by one
    //    16-lane group have 16 different u, hence 16 different instructions.
    //  * B (W2: each of the C output rows contributes its 64 hidden columns of
    //    the step, 128 contiguous bytes): instruction 8 set + i holds, for the
    //    two output blocks 2 set + bb, the rows tau(m) with
    //    m = 16 mhi + 2 i + mlo at slot 4 bb + 2 mhi + mlo.  One 16-lane group
    //    reads 8 instructions x 2 slot parities.  With that numbering
    //    tau(m) = T(i) + 8 mhi + mlo, T(i) = 16 ((i >> 1) & 1) + 4 (i >> 2) + 2 (i & 1),
    //    so the source of a lane is a wave-uniform base plus a lane offset.
    static constexpr int PW = C == 256 ? 8 : 4;            // weight fragments in flight per wave (measured)
    static constexpr int FA = G::NIA / NW;                 // DMA instructions per wave for an A buffer
    static constexpr int FB = G::NIB / NW;                 // ... for a B buffer
    static_assert(G::NIA % NW == 0 && G::NIB % NW == 0, "uniform DMA count per wave");
    static __device__ __forceinline__ uint8_t *buf_a(const Args &a, uint8_t *smem, int slot) {
        return smem + a.off_big + slot * G::BUF_A;
    }
    static __device__ __forceinline__ uint8_t *buf_b(const Args &a, uint8_t *smem, int slot) {
        return smem + a.off_big + 2 * G::BUF_A + slot * G::BUF_B;
    }
    static __device__ __forceinline__ uint32_t t_of(int i) {
        return (uint32_t)(16 * ((i >> 1) & 1) + 4 * (i >> 2) + 2 * (i & 1));
    }
    // lane byte offsets of the sources (A: 16-row group g, piece p; B: slot, piece)
    static __device__ __forceinline__ uint32_t lane_a(int lane) {
        const int per = 64 / RPI, g = lane / per, p = lane % per;
        return (uint32_t)(16 * g * C + 8 * p) * 2;
    }
    static __device__ __forceinline__ uint32_t lane_b(const Args &a, int lane) {
        const int slot = lane >> 3, piece = lane & 7;
        const int bb = slot >> 2, mhi = (slot >> 1) & 1, mlo = slot & 1;
        return ((uint32_t)(32 * bb + 8 * mhi + mlo) * (uint32_t)(a.nch * 32) + 8 * piece) * 2;
    }
    // Wave wv issues instructions I = wv + NW i of every buffer.  With NW = 8
    // and wv < 8, A's instruction I holds W1 row 32 (i >> 1) + 8 (i & 1) + wv
    // of the step and B's holds output rows 64 i + T(wv): the sources are a
    // per-wave base plus compile-time (A) or per-launch (B) offsets, set up
    // once so that a copy costs a few scalar instructions.
    static_assert(NW == 8, "DMA instruction numbering assumes eight waves");
    struct DmaBase {
        const uint8_t *a0;    // W1 row wv (step 0)
        const uint8_t *b0;    // W2 row T(wv), hidden column 0
        uint32_t bstride;     // bytes from W2 row r to row r + 64
        uint32_t lds_a, lds_b;  // LDS address of instruction wv in buffers A0 / B0
    };
    static __device__ __forceinline__ DmaBase dma_base(const Args &a, uint8_t *smem, int wv) {
        const int wu = __builtin_amdgcn_readfirstlane(wv);
        const uint32_t ec = (uint32_t)a.nch * 32;
        DmaBase d;
        d.a0 = reinterpret_cast<const uint8_t *>(a.w1) + (size_t)wu * (C * 2);
        d.b0 = reinterpret_cast<const uint8_t *>(a.w2) + (size_t)t_of(wu) * ec * 2;
        d.bstride = 64u * ec * 2u;
        d.lds_a = lds_addr(buf_a(a, smem, 0)) + (uint32_t)wu * PITCH;
        d.lds_b = lds_addr(buf_b(a, smem, 0)) + (uint32_t)wu * PITCH;
        return d;
    }
    static __device__ __forceinline__ void dma_a(const DmaBase &d, int step, uint32_t la) {
        const uint8_t *src = d.a0 + (size_t)step * (64 * C * 2);
        const uint32_t lds = d.lds_a + (uint32_t)(step & 1) * G::BUF_A;
#pragma unroll
        for (int i = 0; i < FA; i++)
            dma16s_at(src + (32 * (i >> 1) + 8 * (i & 1)) * (C * 2), la, lds + (uint32_t)(i * NW * PITCH));
    }
    static __device__ __forceinline__ void dma_b(const DmaBase &d, int step, uint32_t lb) {
        const uint8_t *src = d.b0 + (size_t)step * 128;
        const uint32_t lds = d.lds_b + (uint32_t)(step & 1) * G::BUF_B;
#pragma unroll
        for (int i = 0; i < FB; i++)
            dma16s_at(src + (size_t)(i * d.bstride), lb, lds + (uint32_t)(i * NW * PITCH));
    }
    // fragment bases of lane (h, m): expand reads W1 row sigma(m) of chunk r
    // (K step ks at +32 ks); project reads output row tau(m) of block cb,
    // hidden columns of chunk j (at a compile-time offset per fragment)
    static __device__ __forceinline__ uint32_t frag_a(int r, int lane) {
        const int h = lane >> 5, rho = sigma_row(lane & 31);
        const int q = 2 * r + (rho >> 4), u = rho & 15;
        return (uint32_t)((u + 16 * (q / RPI)) * PITCH + (q % RPI) * 2 * C + 16 * h);
    }
    static __device__ __forceinline__ uint32_t frag_b(int lane) {
        const int h = lane >> 5, m = lane & 31;
        return (uint32_t)(((m >> 1) & 7) * PITCH + (2 * (m >> 4) + (m & 1)) * 128 + 16 * h);
    }
    static constexpr uint32_t frag_b_off(int cb, int j, int kk) {
        return (uint32_t)((8 * (cb >> 1)) * PITCH + 4 * (cb & 1) * 128 + 64 * j + 32 * kk);
    }

    // ---- halo slab copy (synchronous, through registers): rows of the tile's
    // image rows g_lo - PAD .., channels slab*128 .. +127, pad columns zeroed.
    template <int NTV = NT>
    static __device__ void copy_slab(const Args &a, uint8_t *smem, uint32_t g_lo, int rows, int slab, int tid) {
        const int WP = a.W + 2 * PAD;
        const int per_row = WP * 16;  // 16-byte chunks per halo row
        const int total = rows * per_row;
        const uint8_t *xb = reinterpret_cast<const uint8_t *>(a.x);
        // batches of 8 chunks per thread: all loads of a batch are in flight
        // before the first LDS write
        for (int c0 = 0; c0 < total; c0 += 8 * NTV) {
            u32x4 v[8];
            uint32_t dst[8];
#pragma unroll
            for (int u = 0; u < 8; u++) {
                const int ci = c0 + u * NTV + tid;
                const int r = ci / per_row, rem = ci - r * per_row;
                const int col = rem >> 4, q = rem & 15;
                const int px = col - PAD;
                const int grow = (int)g_lo - PAD + r;
                dst[u] = ci < total ? a.off_big + (uint32_t)r * a.rsl + (uint32_t)col * HPX + q * 16 : 0xffffffffu;
                v[u] = u32x4{0u, 0u, 0u, 0u};
                if (ci < total && px >= 0 && px < a.W && grow >= 0 && grow < a.NH)
                    v[u] = *reinterpret_cast<const u32x4 *>(xb + ((size_t)grow * a.W + px) * (C * 2) + slab * HPX +
                                                            q * 16);
            }
#pragma unroll
            for (int u = 0; u < 8; u++)
                if (dst[u] != 0xffffffffu)
                    *reinterpret_cast<u32x4 *>(smem + dst[u]) = v[u];
        }
    }

    // ---- depth-wise conv of one slab, channel-major.  Lane channel group cq
    // (4 channels) of half-wave hw computes NPX consecutive pixels starting at
    // pixel q0 = q0base + NPX * hw of block b.  All taps of the lane's channels
    // and its s0 / b0 are loaded once (a single round trip), then the tap rows
    // are unrolled so that the LDS reads can run ahead of the FMAs.
    template <int NPX>
    static __device__ void dw_slab(const Args &a, uint8_t *smem, uint32_t g_lo, uint32_t pblk, int b, int q0base,
                                   int slab, int lane) {
        const int hw = lane >> 5, cq = lane & 31;
        const int c0 = slab * CS + 4 * cq;
        const int q0 = q0base + NPX * hw;  // first pixel of this half-wave within the block
        // taps: all at once for k <= 3; for larger k one row at a time, the
        // next row's loads issued before the current row is computed
        constexpr int TR = (KS <= 3 && C < 512) ? KS : 1;  // tap rows held per load batch
        u32x2 wt[2][TR * KS];
#pragma unroll
        for (int t = 0; t < TR * KS; t++)
            wt[0][t] = *reinterpret_cast<const u32x2 *>(a.dw_w + (size_t)t * C + c0);
        half2v s0q[2], b0q[2];
#pragma unroll
        for (int e = 0; e < 2; e++) {
            const int c = c0 + 2 * e;
            s0q[e] = half2v{(_Float16)((a.s0 ? a.s0[c] : 1.0f) * QS), (_Float16)((a.s0 ? a.s0[c + 1] : 1.0f) * QS)};
            b0q[e] = half2v{(_Float16)((a.b0 ? a.b0[c] : 0.0f) * QS), (_Float16)((a.b0 ? a.b0[c + 1] : 0.0f) * QS)};
        }
        uint32_t topleft[NPX];
        int hh[NPX];
        {
            uint32_t p = pblk + q0;
            uint32_t gg = fdiv(p < a.P ? p : 0u, a.divW);
            int wc = (int)(p - gg * (uint32_t)a.W);
            int hr = (int)(gg - fdiv(gg, a.divH) * (uint32_t)a.H);
#pragma unroll
            for (int i = 0; i < NPX; i++, p++) {
                topleft[i] = a.off_big + (gg - g_lo) * a.rsl + (uint32_t)wc * HPX + (uint32_t)cq * 8;
                hh[i] = p < a.P ? hr : -KS - 1;  // invalid pixels read zeros only
                if (++wc == a.W) {
                    wc = 0;
                    gg++;
                    if (++hr == a.H)
                        hr = 0;
                }
            }
        }
        half2v acc[NPX][2];
#pragma unroll
        for (int i = 0; i < NPX; i++)
            acc[i][0] = acc[i][1] = splat2(0.0f);
        auto row = [&](int ti, const u32x2 *w) {
#pragma unroll
            for (int i = 0; i < NPX; i++) {
                const int hr = hh[i] + ti - PAD;
                const uint32_t rb = (hr >= 0 && hr < a.H) ? topleft[i] + (uint32_t)ti * a.rsl : a.off_zero;
#pragma unroll
                for (int tj = 0; tj < KS; tj++) {
                    const u32x2 v = *reinterpret_cast<const u32x2 *>(smem + rb + (uint32_t)tj * HPX);
                    acc[i][0] = __builtin_elementwise_fma(h2(v[0]), h2(w[tj][0]), acc[i][0]);
                    acc[i][1] = __builtin_elementwise_fma(h2(v[1]), h2(w[tj][1]), acc[i][1]);
                }
            }
        };
        if constexpr (TR == KS) {
#pragma unroll
            for (int ti = 0; ti < KS; ti++)
                row(ti, &wt[0][ti * KS]);
        } else {
#pragma unroll 1
            for (int ti = 0; ti < KS; ti += 2) {
                if (ti + 1 < KS) {
#pragma unroll
                    for (int tj = 0; tj < KS; tj++)
                        wt[1][tj] = *reinterpret_cast<const u32x2 *>(a.dw_w + (size_t)((ti + 1) * KS + tj) * C + c0);
                }
                row(ti, wt[0]);
                if (ti + 1 < KS) {
                    if (ti + 2 < KS) {
#pragma unroll
                        for (int tj = 0; tj < KS; tj++)
                            wt[0][tj] = *reinterpret_cast<const u32x2 *>(a.dw_w + (size_t)((ti + 2) * KS + tj) * C + c0);
                    }
                    row(ti + 1, wt[1]);
                }
            }
        }
        const uint32_t dbase = a.off_d + (uint32_t)(32 * b + q0) * DPX + (uint32_t)(4 * cq) * 2;
#pragma unroll
        for (int i = 0; i < NPX; i++) {
            u32x2 d;
            d[0] = u32(__builtin_elementwise_fma(acc[i][0], s0q[0], b0q[0]));
            d[1] = u32(__builtin_elementwise_fma(acc[i][1], s0q[1], b0q[1]));
            *reinterpret_cast<u32x2 *>(smem + dbase + (uint32_t)i * DPX) = d;
        }
    }

    // ---- FFN for block b of the tile by wave r of its pair; dfr = D as B
    // fragments, acc = this wave's half of the output channels.
    static __device__ void ffn(const Args &a, uint8_t *smem, int tid, int lane, int b, int r,
                               const u32x4 (&dfr)[KST], float16v (&acc)[CBH]) {
        const int h = lane >> 5;
        const int nsteps = a.nch / 2;
        const int wv = tid >> 6;
        uint8_t *gmine = smem + a.off_g + (uint32_t)(b * 2 + r) * 2048;
        // prologue: A0 B0 A1 B1 in flight; A0 and B0 must land
        const uint32_t la = lane_a(lane), lb = lane_b(a, lane);
        const DmaBase db = dma_base(a, smem, wv);
        dma_a(db, 0, la);
        dma_b(db, 0, lb);
        if (nsteps > 1) {
            dma_a(db, 1, la);
            dma_b(db, 1, lb);
            fused::wait_vmcnt<FA + FB>();
        } else {
            fused::wait_vmcnt<0>();
        }
        lds_barrier();
#pragma unroll 1
        for (int s = 0; s < nsteps; s++) {
            uint8_t *bufa = buf_a(a, smem, s & 1);
            uint8_t *bufb = buf_b(a, smem, s & 1);
            // B_(s+1) goes into the slot B_(s-1) used, free since the last
            // barrier; issued first, so that the copies run beside the MFMAs
            if (s >= 1 && s + 1 < nsteps)
                dma_b(db, s + 1, lb);
            // ---- expand chunk 2s + r: U/4 = s1 * (W1 D/4) + b1/4, phi, hidden tile to LDS
            const int ch = 2 * s + r;
            const uint8_t *wa = bufa + frag_a(r, lane);
            // fragments stream through a PW-deep register window; the
            // scheduling groups keep PW LDS reads in flight ahead of the MFMAs
            // (LDS latency with eight waves reading far exceeds one MFMA)
            float16v hh;
#pragma unroll
            for (int e = 0; e < 16; e++)
                hh[e] = 0.0f;
            u32x4 wf[PW];
#pragma unroll
            for (int i = 0; i < PW; i++)
                wf[i] = ld16(wa, i * 32);
#pragma unroll
            for (int ks = 0; ks < KST; ks++) {
                hh = mfma32(wf[ks % PW], dfr[ks], hh, F16{});
                if (ks + PW < KST)
                    wf[ks % PW] = ld16(wa, (ks + PW) * 32);
            }
            __builtin_amdgcn_sched_group_barrier(0x100, PW, 1);
#pragma unroll
            for (int ks = 0; ks + PW < KST; ks++) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 1);
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 1);
            }
            __builtin_amdgcn_sched_group_barrier(0x008, PW, 1);
            const float16v s1v = *reinterpret_cast<const float16v *>(smem + a.off_s1 + ch * 128 + h * 64);
            const float16v b1v = *reinterpret_cast<const float16v *>(smem + a.off_b1 + ch * 128 + h * 64);
            float v[16];
#pragma unroll
            for (int e = 0; e < 16; e++)
                v[e] = fmaf(hh[e], s1v[e], b1v[e]);
            uint32_t o[8];
            activate<8>(v, o);
            *reinterpret_cast<u32x4 *>(gmine + lane * 32) = u32x4{o[0], o[1], o[2], o[3]};
            *reinterpret_cast<u32x4 *>(gmine + lane * 32 + 16) = u32x4{o[4], o[5], o[6], o[7]};
            // B_s landed (issued after it: A_(s+1), B_(s+1) when they exist)
            if (s + 1 < nsteps)
                fused::wait_vmcnt<FA + FB>();
            else
                fused::wait_vmcnt<0>();
            lds_barrier();  // hidden tiles and B_s visible; A_s free
            // A_(s+2) goes into A_s's slot
            if (s + 2 < nsteps)
                dma_a(db, s + 2, la);
            // ---- project both chunks onto this wave's output half
            {
                constexpr int NF = 4 * CBH;  // W2 fragments used by this wave per step
                u32x4 hid[2][2];
#pragma unroll
                for (int j = 0; j < 2; j++) {
                    const uint8_t *gp = smem + a.off_g + (uint32_t)(b * 2 + j) * 2048 + lane * 32;
                    hid[j][0] = ld16(gp, 0);
                    hid[j][1] = ld16(gp, 16);
                }
                // MFMA i: chunk j = i / (2*CBH), K step kk = (i / CBH) % 2, output block
                // c = i % CBH -- consecutive MFMAs feed different accumulators
                // block cb = CBH r + c (CBH even): set CBH r / 2 + c / 2, bb = c % 2
                static_assert(CBH % 2 == 0, "output blocks in pairs");
                const uint8_t *wb = bufb + frag_b(lane) + (uint32_t)(4 * CBH * r * PITCH);
                auto frag = [&](int i) {
                    const int j = i / (2 * CBH), kk = (i / CBH) & 1, c = i % CBH;
                    return ld16(wb, frag_b_off(c, j, kk));
                };
                u32x4 wf[PW];
#pragma unroll
                for (int i = 0; i < PW; i++)
                    wf[i] = frag(i);
#pragma unroll
                for (int i = 0; i < NF; i++) {
                    const int j = i / (2 * CBH), kk = (i / CBH) & 1, c = i % CBH;
                    acc[c] = mfma32(wf[i % PW], hid[j][kk], acc[c], F16{});
                    if (i + PW < NF)
                        wf[i % PW] = frag(i + PW);
                }
                __builtin_amdgcn_sched_group_barrier(0x100, PW + 4, 2);
#pragma unroll
                for (int i = 0; i + PW < NF; i++) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 2);
                    __builtin_amdgcn_sched_group_barrier(0x100, 1, 2);
                }
                __builtin_amdgcn_sched_group_barrier(0x008, PW, 2);
            }
            // A_(s+1) landed (issued after it: B_(s+1), and A_(s+2) when it exists)
            if (s + 2 < nsteps)
                fused::wait_vmcnt<FB + FA>();
            else if (s + 1 < nsteps)
                fused::wait_vmcnt<FB>();
            lds_barrier();  // B_s and the hidden tiles are free; A_(s+1) visible
        }
        __syncthreads();  // the weight buffers (halo region) are free for the next tile
    }

    static __device__ void run(const Args &a, uint8_t *smem) {
        const int tid = threadIdx.x;
        const int lane = tid & 63, wv = tid >> 6;
        const int h = lane >> 5, m = lane & 31;

        const int Gn = gridDim.x;
        const int g = (Gn % 8 == 0) ? (blockIdx.x % 8) * (Gn / 8) + blockIdx.x / 8 : blockIdx.x;
        const int lo = g * a.range_base + (g < a.range_extra ? g : a.range_extra);
        const int hi = lo + a.range_base + (g < a.range_extra ? 1 : 0);

        for (uint32_t i = a.off_zero / 16 + tid; i < (a.off_zero + KS * HPX + 64) / 16; i += NT)
            reinterpret_cast<u32x4 *>(smem)[i] = u32x4{0u, 0u, 0u, 0u};
        stage_vectors(a, smem, tid);

        const int b = wv & (NBLK - 1), r = wv >> 2;  // block of the tile, role in its pair
        for (int t0 = lo; t0 < hi; t0 += NBLK) {
            const int nblk = hi - t0 < NBLK ? hi - t0 : NBLK;
            const uint32_t p0 = (uint32_t)t0 * 32;
            uint32_t pend = p0 + (uint32_t)nblk * 32;
            if (pend > a.P)
                pend = a.P;
            const uint32_t g_lo = fdiv(p0, a.divW);
            const int rows = (int)(fdiv(pend - 1, a.divW) - g_lo) + 1 + 2 * PAD;
            const bool mine = b < nblk;
            const uint32_t pblk = p0 + 32u * b;

            u32x4 dfr[KST];
#pragma unroll
            for (int slab = 0; slab < NSLAB; slab++) {
                __syncthreads();  // halo / D buffers free
                copy_slab(a, smem, g_lo, rows, slab, tid);
                __syncthreads();
                if (mine)
                    dw_slab<8>(a, smem, g_lo, pblk, b, 16 * r, slab, lane);
                __syncthreads();
#pragma unroll
                for (int k8 = 0; k8 < CS / 16; k8++)
                    dfr[slab * (CS / 16) + k8] =
                        ld16(smem, a.off_d + (uint32_t)(32 * b + m) * DPX + (uint32_t)(k8 * 16 + 8 * h) * 2);
            }
            __syncthreads();  // D and halo reads done before the weight buffers overwrite them

            float16v acc[CBH];
#pragma unroll
            for (int c = 0; c < CBH; c++)
#pragma unroll
                for (int e = 0; e < 16; e++)
                    acc[c][e] = 0.0f;
            ffn(a, smem, tid, lane, b, r, dfr, acc);

            // epilogue: y = x + 4 * acc + b2 on this wave's output half
            const uint32_t pix = pblk + m;
            if (mine && pix < a.P) {
#pragma unroll
                for (int c = 0; c < CBH; c++) {
                    const int cc = (r * CBH + c) * 32 + 16 * h;
                    const float16v sv = *reinterpret_cast<const float16v *>(smem + a.off_s2b2 + cc * 4);
                    const float16v bv = *reinterpret_cast<const float16v *>(smem + a.off_s2b2 + 4 * C + cc * 4);
                    const u32x4 *xs = reinterpret_cast<const u32x4 *>(a.x + (size_t)pix * C + cc);
                    Pack8 x0, x1;
                    x0.u = xs[0];
                    x1.u = xs[1];
                    u32x4 o0, o1;
#pragma unroll
                    for (int q = 0; q < 4; q++) {
                        o0[q] = F16::pack2(fmaf(acc[c][2 * q], sv[2 * q], F16::lo(x0.w[q]) + bv[2 * q]),
                                           fmaf(acc[c][2 * q + 1], sv[2 * q + 1], F16::hi(x0.w[q]) + bv[2 * q + 1]));
                        o1[q] = F16::pack2(fmaf(acc[c][8 + 2 * q], sv[8 + 2 * q], F16::lo(x1.w[q]) + bv[8 + 2 * q]),
                                           fmaf(acc[c][8 + 2 * q + 1], sv[8 + 2 * q + 1], F16::hi(x1.w[q]) + bv[8 + 2 * q + 1]));
                    }
                    u32x4 *dst = reinterpret_cast<u32x4 *>(a.y + (size_t)pix * C + cc);
                    dst[0] = o0;
                    dst[1] = o1;
                }
            }
        }
    }
};

// ---------------------------------------------------------------------------
// C = 512: one wave per 32-pixel block (4 waves, one per SIMD, 512 registers
// each: the 512-channel accumulators of a block alone take 256).  The FFN
// walks the hidden chunks of its group one at a time; W1 and W2 fragments of
// a chunk (64 KB) stream through a two-slot LDS ring by asynchronous copies
// issued one chunk ahead.  With grid.y > 1 the hidden chunks are split over
// workgroups: each writes 4 s2 W2 phi(U) of its chunks as an fp32 partial and
// a second kernel adds the partials in group order, b2 and x.
struct SoloArgs {
    Args a;
    float *partial;  // [groups][P][C] fp32, or nullptr (one group: write y)
    int chunks_per_group;
    int ntiles;
};

template <int C, int KS, int ACT>
struct Ks {
    static constexpr int NWS = 4, NTS = NWS * 64;
    typedef Kw<C, KS, ACT> K;
    static constexpr int KST = C / 16, CB = C / 32, NSLAB = C / CS;
    // One chunk of weights in LDS, filled by LDS-DMA instructions of 1 KB each
    // that read contiguous memory; every instruction's KB sits at a pitch of
    // PITCH bytes (16 bytes of padding), which makes the A-fragment reads
    // below hit 16 different bank groups per 16 lanes:
    //  * W1 (rows of C halves, contiguous in memory): C = 512: instruction j
    //    copies row j; C = 256: instruction j copies rows j and j + 16 (the two
    //    rows are read by different 16-lane groups).  The expand fragment of K
    //    step ks, lane (h, m), is row sigma(m), bytes 32 ks + 16 h.
    //  * W2: each of the C rows contributes 64 contiguous bytes (its 32 hidden
    //    columns).  Output blocks are taken four at a time; within such a set,
    //    instruction i (0..7) holds, for each of the four blocks, the rows
    //    tau(m) with m = 4i .. 4i+3, at slot 4 * block + m % 4.  The project
    //    fragment (cb, kk), lane (h, m), is then at
    //    (cb/4)*8*PITCH + (m/4)*PITCH + (cb%4)*256 + (m%4)*64 + 32 kk + 16 h.
    static constexpr int PITCH = 1040;
    static constexpr int RPI = 1024 / (2 * C);           // W1 rows per instruction
    static constexpr int NI1 = 32 / RPI, NI2 = 2 * CB;    // instructions per chunk
    static constexpr int W2OFF = NI1 * PITCH;
    static constexpr int SLOT = W2OFF + NI2 * PITCH;
    static_assert((C == 512 || C == 256) && CB % 4 == 0, "solo kernel: C = 256 or 512");
    static constexpr int WIN = C == 512 ? 4 : 8;  // fragment reads in flight (registers permitting)

    // LDS offset of W1 row r inside a chunk slot
    static __device__ __forceinline__ uint32_t w1_row(int r) {
        return RPI == 1 ? (uint32_t)r * PITCH : (uint32_t)(r & 15) * PITCH + (uint32_t)(r >> 4) * (2 * C);
    }

    // This wave's 1 KB pieces of a chunk: NPW copies.  The source of a
    // lane's 16 bytes in piece q is a wave-uniform base (piece_base) plus a
    // per-lane byte offset that depends only on the kind of piece (lane_offs).
    static constexpr int NPW = (NI1 + NI2) / NWS;
    struct LaneOffs {
        uint32_t w1, w2;
    };
    static __device__ __forceinline__ LaneOffs lane_offs(const Args &a, int lane) {
        LaneOffs o;
        // W1: lane -> row 16 * (lane / 32) of the instruction's pair (C = 256), piece lane % (64 / RPI)
        const int lr = RPI == 1 ? 0 : 16 * (lane >> 5), lp = RPI == 1 ? lane : (lane & 31);
        o.w1 = (uint32_t)(lr * C + 8 * lp) * 2;
        // W2: lane -> slot s = lane / 4 (block bq = s / 4 of the set, row m % 4 = s % 4), piece lane % 4;
        // with m = 4 i + s % 4, tau(m) = 16 (i & 1) + 4 (i >> 1) + s % 4
        const int sl = lane >> 2, bq = sl >> 2, r4 = sl & 3, pc = lane & 3;
        o.w2 = ((uint32_t)(32 * bq + r4) * (uint32_t)(a.nch * 32) + 8 * pc) * 2;
        return o;
    }
    // Wave wv copies pieces q = 0 .. NPW - 1: W1 instruction j = wv + NWS q
    // (rows ch*32 + j), then W2 instruction j = wv + NWS q' (q' = q - NI1/NWS)
    // with set st = j >> 3 and index i = j & 7, that is output rows
    // 128 st + 16 (i & 1) + 4 (i >> 1) = R(wv) + 128 (q' >> 1) + 8 (q' & 1),
    // R(wv) = 16 (wv & 1) + 4 (wv >> 1) (NWS = 4, wv < 4).  The per-wave
    // bases are set up once; a piece adds a compile-time or per-launch offset.
    static_assert(NWS == 4, "piece numbering assumes four waves");
    struct CopyBase {
        const uint8_t *w1, *w2;  // W1 row wv, W2 row R(wv) (chunk 0)
        uint32_t e2;             // bytes per W2 row
        uint32_t lds;            // LDS address of instruction wv in slot 0
    };
    static __device__ __forceinline__ CopyBase copy_base(const Args &a, uint8_t *smem, int wv) {
        const int wu = __builtin_amdgcn_readfirstlane(wv);
        CopyBase cb;
        cb.e2 = (uint32_t)a.nch * 64;
        cb.w1 = reinterpret_cast<const uint8_t *>(a.w1) + (size_t)wu * (C * 2);
        cb.w2 = reinterpret_cast<const uint8_t *>(a.w2) + (size_t)(16 * (wu & 1) + 4 * (wu >> 1)) * cb.e2;
        cb.lds = lds_addr(smem + a.off_big) + (uint32_t)wu * PITCH;
        return cb;
    }
    // pieces Q0 .. Q1-1 of this wave's copies of chunk ch (W1 pieces first)
    template <int Q0 = 0, int Q1 = NPW>
    static __device__ __forceinline__ void dma_chunk(const CopyBase &cb, int ch, int slot, const LaneOffs &lo) {
        const uint8_t *s1 = cb.w1 + (size_t)ch * (32 * C * 2);
        const uint8_t *s2 = cb.w2 + (size_t)ch * 64;
        const uint32_t lds = cb.lds + (uint32_t)slot * SLOT;
#pragma unroll
        for (int q = Q0; q < Q1; q++) {
            if (q < NI1 / NWS) {
                dma16s_at(s1 + q * NWS * (C * 2), lo.w1, lds + (uint32_t)(q * NWS * PITCH));
            } else {
                const int qq = q - NI1 / NWS;
                dma16s_at(s2 + (size_t)((uint32_t)(128 * (qq >> 1) + 8 * (qq & 1)) * cb.e2), lo.w2,
                          lds + (uint32_t)(W2OFF + qq * NWS * PITCH));
            }
        }
    }
    static __device__ void run(const SoloArgs &sa, uint8_t *smem) {
        const Args &a = sa.a;
        const int tid = threadIdx.x;
        const int lane = tid & 63, wv = tid >> 6;
        const int h = lane >> 5, m = lane & 31;
        const int grp = blockIdx.y;
        const int ch0 = grp * sa.chunks_per_group, nchg = sa.chunks_per_group;
        const LaneOffs lofs = lane_offs(a, lane);
        const CopyBase cpb = copy_base(a, smem, wv);

        for (uint32_t i = a.off_zero / 16 + tid; i < (a.off_zero + KS * HPX + 64) / 16; i += NTS)
            reinterpret_cast<u32x4 *>(smem)[i] = u32x4{0u, 0u, 0u, 0u};
        K::template stage_vectors<NTS>(a, smem, tid, ch0, nchg);

        for (int tile = blockIdx.x; tile < sa.ntiles; tile += gridDim.x) {
            const uint32_t p0 = (uint32_t)tile * 128;
            uint32_t pend = p0 + 128;
            if (pend > a.P)
                pend = a.P;
            const uint32_t g_lo = fdiv(p0, a.divW);
            const int rows = (int)(fdiv(pend - 1, a.divW) - g_lo) + 1 + 2 * K::PAD;
            const uint32_t pblk = p0 + 32u * wv;
            const bool mine = pblk < a.P;

            u32x4 dfr[KST];
#pragma unroll
            for (int slab = 0; slab < NSLAB; slab++) {
                __syncthreads();
                K::template copy_slab<NTS>(a, smem, g_lo, rows, slab, tid);
                __syncthreads();
                if (mine) {
                    // 16 pixels per half-wave; 8 at a time where registers are short
                    if constexpr (KS >= 7 || C == 512) {
                        K::template dw_slab<8>(a, smem, g_lo, pblk, wv, 0, slab, lane);
                        K::template dw_slab<8>(a, smem, g_lo, pblk, wv, 16, slab, lane);
                    } else {
                        K::template dw_slab<16>(a, smem, g_lo, pblk, wv, 0, slab, lane);
                    }
                }
                __syncthreads();
#pragma unroll
                for (int k8 = 0; k8 < CS / 16; k8++)
                    dfr[slab * (CS / 16) + k8] =
                        ld16(smem, a.off_d + (uint32_t)(32 * wv + m) * DPX + (uint32_t)(k8 * 16 + 8 * h) * 2);
            }
            __syncthreads();  // D and halo reads done before the ring overwrites them

            float16v acc[CB];
#pragma unroll
            for (int c = 0; c < CB; c++)
#pragma unroll
                for (int e = 0; e < 16; e++)
                    acc[c][e] = 0.0f;

            dma_chunk(cpb, ch0, 0, lofs);
#pragma unroll 1
            for (int c = 0; c < nchg; c++) {
                fused::wait_vmcnt<0>();  // this wave's copies of chunk c have landed
                lds_barrier();           // everyone's have; the other slot is free
                // the next chunk's copies in two halves (W1 now, W2 before the
                // project), so that each burst fits the copy queue and drains
                // beside the MFMAs instead of holding the wave at issue
                if (c + 1 < nchg)
                    dma_chunk<0, NPW / 2>(cpb, ch0 + c + 1, (c + 1) & 1, lofs);
                const uint8_t *slot = smem + a.off_big + (c & 1) * SLOT;
                const uint8_t *f1 = slot + w1_row(sigma_row(m)) + h * 16;
                const uint8_t *f2 = slot + W2OFF + (m >> 2) * PITCH + (m & 3) * 64 + h * 16;
                // expand (4-deep fragment window)
                float16v hh;
#pragma unroll
                for (int e = 0; e < 16; e++)
                    hh[e] = 0.0f;
                u32x4 wf[WIN];
#pragma unroll
                for (int i = 0; i < WIN; i++)
                    wf[i] = ld16(f1, i * 32);
#pragma unroll
                for (int ks = 0; ks < KST; ks++) {
                    hh = mfma32(wf[ks % WIN], dfr[ks], hh, F16{});
                    if (ks + WIN < KST)
                        wf[ks % WIN] = ld16(f1, (ks + WIN) * 32);
                }
                __builtin_amdgcn_sched_group_barrier(0x100, WIN, 1);
#pragma unroll
                for (int ks = 0; ks + WIN < KST; ks++) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 1);
                    __builtin_amdgcn_sched_group_barrier(0x100, 1, 1);
                }
                __builtin_amdgcn_sched_group_barrier(0x008, WIN, 1);
                const float16v s1v = *reinterpret_cast<const float16v *>(smem + a.off_s1 + c * 128 + h * 64);
                const float16v b1v = *reinterpret_cast<const float16v *>(smem + a.off_b1 + c * 128 + h * 64);
                float v[16];
#pragma unroll
                for (int e = 0; e < 16; e++)
                    v[e] = fmaf(hh[e], s1v[e], b1v[e]);
                uint32_t o[8];
                K::template activate<8>(v, o);
                const u32x4 hid[2] = {u32x4{o[0], o[1], o[2], o[3]}, u32x4{o[4], o[5], o[6], o[7]}};
                // project: MFMA i -> K step kk = i / CB, output block i % CB
                // W2 fragment (cb, kk) of MFMA i: cb = i % CB, kk = i / CB
                auto w2off = [](int i) {
                    const int cb = i % CB, kk = i / CB;
                    return (uint32_t)((cb >> 2) * 8 * PITCH + (cb & 3) * 256 + kk * 32);
                };
                if (c + 1 < nchg)
                    dma_chunk<NPW / 2, NPW>(cpb, ch0 + c + 1, (c + 1) & 1, lofs);
#pragma unroll
                for (int i = 0; i < WIN; i++)
                    wf[i] = ld16(f2, w2off(i));
#pragma unroll
                for (int i = 0; i < 2 * CB; i++) {
                    acc[i % CB] = mfma32(wf[i % WIN], hid[i / CB], acc[i % CB], F16{});
                    if (i + WIN < 2 * CB)
                        wf[i % WIN] = ld16(f2, w2off(i + WIN));
                }
                __builtin_amdgcn_sched_group_barrier(0x100, WIN, 2);
#pragma unroll
                for (int i = 0; i + WIN < 2 * CB; i++) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 2);
                    __builtin_amdgcn_sched_group_barrier(0x100, 1, 2);
                }
                __builtin_amdgcn_sched_group_barrier(0x008, WIN, 2);
            }
            __syncthreads();  // the ring is free for the next tile

            const uint32_t pix = pblk + m;
            if (mine && pix < a.P) {
#pragma unroll
                for (int cb = 0; cb < CB; cb++) {
                    const int cc = cb * 32 + 16 * h;
                    const float16v sv = *reinterpret_cast<const float16v *>(smem + a.off_s2b2 + cc * 4);
                    if (sa.partial) {
                        float4v *dst = reinterpret_cast<float4v *>(sa.partial + ((size_t)grp * a.P + pix) * C + cc);
#pragma unroll
                        for (int q = 0; q < 4; q++)
                            dst[q] = float4v{acc[cb][4 * q] * sv[4 * q], acc[cb][4 * q + 1] * sv[4 * q + 1],
                                             acc[cb][4 * q + 2] * sv[4 * q + 2], acc[cb][4 * q + 3] * sv[4 * q + 3]};
                    } else {
                        const float16v bv = *reinterpret_cast<const float16v *>(smem + a.off_s2b2 + 4 * C + cc * 4);
                        const u32x4 *xs = reinterpret_cast<const u32x4 *>(a.x + (size_t)pix * C + cc);
                        Pack8 x0, x1;
                        x0.u = xs[0];
                        x1.u = xs[1];
                        u32x4 o0, o1;
#pragma unroll
                        for (int q = 0; q < 4; q++) {
                            o0[q] = F16::pack2(fmaf(acc[cb][2 * q], sv[2 * q], F16::lo(x0.w[q]) + bv[2 * q]),
                                               fmaf(acc[cb][2 * q + 1], sv[2 * q + 1], F16::hi(x0.w[q]) + bv[2 * q + 1]));
                            o1[q] = F16::pack2(
                                fmaf(acc[cb][8 + 2 * q], sv[8 + 2 * q], F16::lo(x1.w[q]) + bv[8 + 2 * q]),
                                fmaf(acc[cb][8 + 2 * q + 1], sv[8 + 2 * q + 1], F16::hi(x1.w[q]) + bv[8 + 2 * q + 1]));
                        }
                        u32x4 *dst = reinterpret_cast<u32x4 *>(a.y + (size_t)pix * C + cc);
                        dst[0] = o0;
                        dst[1] = o1;
                    }
                }
            }
        }
    }
};

template <int C, int KS, int ACT>
__global__ __launch_bounds__(256, 1) void solo_kernel(SoloArgs sa) {
    extern __shared__ __attribute__((aligned(256))) uint8_t smem[];
    Ks<C, KS, ACT>::run(sa, smem);
}

template <int C, int KS, int ACT>
__global__ __launch_bounds__(NT, 1) void wide_kernel(Args a) {
    extern __shared__ __attribute__((aligned(256))) uint8_t smem[];
    Kw<C, KS, ACT>::run(a, smem);
}

template <int C, int KS>
hipError_t launch_ck(const void *x, void *y, const BlockW &w, const Shape &s, hipStream_t st) {
    const int pad = KS / 2;
    const int64_t NH = (int64_t)s.N * s.H;
    const int halo_rows = halo_rows_for(KS, s.W, NH);
    const uint32_t rsl = (uint32_t)(s.W + 2 * pad) * HPX;
    const int nch = s.E * C / 32;
    const Layout L = layout_for<C>(nch, KS, halo_rows, rsl);
    if (L.total > 160 * 1024)
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
    a.nch = nch;
    const int64_t P = (int64_t)s.N * s.H * s.W;
    a.P = (uint32_t)P;
    a.divW = fused::make_fastdiv((uint32_t)s.W);
    a.divH = fused::make_fastdiv((uint32_t)s.H);
    const int nblocks = (int)((P + 31) / 32);
    int Gn = device_cu_count();
    if (Gn > nblocks)
        Gn = nblocks;
    a.range_base = nblocks / Gn;
    a.range_extra = nblocks % Gn;
    a.rsl = rsl;
    a.off_b1 = L.b1;
    a.off_g = L.g;
    a.off_s1 = L.s1;
    a.off_s2b2 = L.s2b2;
    a.off_d = L.d;
    a.off_big = L.big;
    a.off_zero = L.zero;
    hipError_t e;
#define CF_WIDE_LAUNCH(ACTV)                                                                                         \
    {                                                                                                                 \
        auto kf = wide_kernel<C, KS, ACTV>;                                                                          \
        if ((e = allow_full_lds((const void *)kf))) \
            return e;                                                                                                 \
        hipLaunchKernelGGL(kf, dim3(Gn), dim3(NT), L.total, st, a);                                                  \
    }
    switch (s.act) {
    case ACT_GELU: CF_WIDE_LAUNCH(ACT_GELU) break;
    case ACT_RELU: CF_WIDE_LAUNCH(ACT_RELU) break;
    default: CF_WIDE_LAUNCH(ACT_NONE) break;
    }
#undef CF_WIDE_LAUNCH
    return hipGetLastError();
}

template <int C>
hipError_t launch_c(const void *x, void *y, const BlockW &w, const Shape &s, hipStream_t st) {
    switch (s.k) {
    case 1: return launch_ck<C, 1>(x, y, w, s, st);
    case 3: return launch_ck<C, 3>(x, y, w, s, st);
    case 5: return launch_ck<C, 5>(x, y, w, s, st);
    default: return launch_ck<C, 7>(x, y, w, s, st);
    }
}

// C = 512 launcher.  groups > 1 requires `partial` ([groups][P][C] fp32); the
// caller then runs the ordered reduction.
template <int C, int KS>
hipError_t launch_solo(const void *x, void *y, const BlockW &w, const Shape &s, int groups, float *partial,
                       hipStream_t st) {
    const int pad = KS / 2;
    const int nch = s.E * C / 32;
    if (groups < 1 || nch % groups)
        return hipErrorInvalidValue;
    const int nchg = nch / groups;
    const int64_t NH = (int64_t)s.N * s.H;
    const int halo_rows = halo_rows_for(KS, s.W, NH);
    const uint32_t rsl = (uint32_t)(s.W + 2 * pad) * HPX;
    // [b1 regs][s1 regs][4 s2 | b2][overlay: halo + D | ring of two chunks][zero]
    Layout L;
    L.b1 = 0;
    L.s1 = (uint32_t)nchg * 128;
    L.s2b2 = L.s1 + (uint32_t)nchg * 128;
    L.g = 0;
    L.big = (L.s2b2 + C * 8 + 255) & ~255u;
    L.d = L.big + (((uint32_t)halo_rows * rsl + 255) & ~255u);
    const uint32_t hd = (L.d - L.big) + NBLK * 32 * DPX;
    const uint32_t ring = 2u * Ks<C, KS, ACT_NONE>::SLOT;
    L.zero = L.big + (hd > ring ? hd : ring);
    L.total = L.zero + (uint32_t)KS * HPX + 64;
    if (L.total > 160 * 1024)
        return hipErrorInvalidConfiguration;
    SoloArgs sa{};
    Args &a = sa.a;
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
    a.nch = nch;
    const int64_t P = (int64_t)s.N * s.H * s.W;
    a.P = (uint32_t)P;
    a.divW = fused::make_fastdiv((uint32_t)s.W);
    a.divH = fused::make_fastdiv((uint32_t)s.H);
    a.rsl = rsl;
    a.off_b1 = L.b1;
    a.off_s1 = L.s1;
    a.off_s2b2 = L.s2b2;
    a.off_g = L.g;
    a.off_d = L.d;
    a.off_big = L.big;
    a.off_zero = L.zero;
    sa.partial = groups > 1 ? partial : nullptr;
    sa.chunks_per_group = nchg;
    sa.ntiles = (int)((P + 127) / 128);
    const int cus = device_cu_count();
    int gx = (cus + groups - 1) / groups;
    if (gx > sa.ntiles)
        gx = sa.ntiles;
    hipError_t e;
#define CF_SOLO_LAUNCH(ACTV)                                                                                         \
    {                                                                                                                 \
        auto kf = solo_kernel<C, KS, ACTV>;                                                                             \
        if ((e = allow_full_lds((const void *)kf))) \
            return e;                                                                                                 \
        hipLaunchKernelGGL(kf, dim3(gx, groups), dim3(256), L.total, st, sa);                                       \
    }
    switch (s.act) {
    case ACT_GELU: CF_SOLO_LAUNCH(ACT_GELU) break;
    case ACT_RELU: CF_SOLO_LAUNCH(ACT_RELU) break;
    default: CF_SOLO_LAUNCH(ACT_NONE) break;
    }
#undef CF_SOLO_LAUNCH
    return hipGetLastError();
}

inline hipError_t launch_c512(const void *x, void *y, const BlockW &w, const Shape &s, int groups, float *partial,
                              hipStream_t st) {
    switch (s.k) {
    case 1: return launch_solo<512, 1>(x, y, w, s, groups, partial, st);
    case 3: return launch_solo<512, 3>(x, y, w, s, groups, partial, st);
    case 5: return launch_solo<512, 5>(x, y, w, s, groups, partial, st);
    default: return launch_solo<512, 7>(x, y, w, s, groups, partial, st);
    }
}

}  // namespace wide

hipError_t launch_wide_c128(const void *x, void *y, const BlockW &w, const Shape &s, hipStream_t st);
hipError_t launch_wide_c256(const void *x, void *y, const BlockW &w, const Shape &s, hipStream_t st);
hipError_t launch_wide_c512(const void *x, void *y, const BlockW &w, const Shape &s, int groups, float *partial,
                            hipStream_t st);

}  // namespace cf
