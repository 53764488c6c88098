// cf_gblock.h -- fused ConvFirst block with the paper's own first layer: a
// 3 x 3 grouped convolution of group width 8 (Sec. 5.3 of Lavin,
// arXiv:2404.03617, eq. f:grouped-conv2d with K = C, T = 8), then the FFN
// (expand, activation, project) in the loop-fused order of eq. e:ffn-eff, and
// the residual shortcut; batch norms folded to per-channel scale and bias.
// Instantiated per channel count in cf_gblock_c*.hip.
//
// Work unit: a block of 4 image rows x 16 columns (64 pixels) of one image.
// A workgroup of NW waves runs NW blocks at a time, one per wave; each wave
// keeps its own halo (6 rows x 18 columns) in a private LDS region.  Four
// rows per wave halve the LDS reads of the FFN weights per pixel against two
// rows (every weight fragment read feeds four products).  The FFN
// weights are either resident in LDS for the whole kernel (when every chunk
// of 32 hidden channels fits beside the halos: no barrier after the start)
// or stream through a two-slot LDS ring, one chunk per workgroup barrier,
// each chunk's global loads issued two chunks before it is needed.
//
// All products are v_mfma_f32_16x16x32 (fp16 or bf16 in, fp32 accumulate).
// Layouts (lane l, q = l >> 4, j = l & 15): A row j, k = 8q..8q+7; B column j,
// k = 8q..8q+7; D column j, rows 4q..4q+3.
//
//  * Grouped conv on the matrix unit.  For group g (channels 8g..8g+7) and
//    the block's row pair p, one 16 x 16 x 32 product per tap column dj
//    evaluates 16 output pixels x 2 rows at once: D row m = 8s + o is output
//    channel 8g + o of block row 2p + s, D column j is block column j, and
//    the K index is (tap row R of the 4-row halo window starting at halo row
//    2p, input channel t) -- B lane (j, q) reads halo pixel (row 2p + q,
//    column j + dj), channels 8g..8g+7, one 16-byte LDS read; A row
//    (s, o) at (R, t) is the tap W[R - s][dj][8g + o][t], zero when R - s is
//    outside 0..2.  Three products per group cover the 3 x 3 taps; 72 of
//    every 96 multiply-adds are useful (a block-diagonal product with 16
//    output channels and 16 input channels per step would use 50% or less).
//  * The conv output d = s0 * conv + b0, rounded to the I/O dtype, goes to the
//    wave's LDS region and comes back as the expand's B fragments, read once
//    per block and kept in registers for every hidden chunk.  Group g's d
//    values overwrite only the bytes of its own 8 channels, which later
//    groups do not read, and row pair 0's d (pixels 0..31 of the region)
//    lies below the halo rows row pair 1 reads (pixels 36 on), so they are
//    stored as soon as they are computed.
//  * Expand: two 16-row products per chunk and K step, with the W1 rows of a
//    chunk ordered so that expand tile t row m is hidden channel
//    8 (m >> 2) + 4 t + (m & 3): lane group q then holds hidden channels
//    8q..8q+7 -- exactly the B fragment of the project product, which needs
//    no data movement.  s1, b1 and the activation are applied in fp32, the
//    result rounded to the I/O dtype.
//  * Project: C/16 products per chunk into fp32 accumulators; the epilogue
//    adds s2, b2 and the block input x -- read from the halo's centre pixels
//    at the start of the block, before the conv outputs overwrite them, and
//    kept in registers (a global re-read at the end would stall every block
//    on a full memory latency) -- and stores the output once.
//  * Halo prefetch.  With few channels (PREF2) a block's halo is loaded into
//    registers a whole block ahead: when block r's D fragments are in
//    registers, the halo of block r+1 (loaded during block r-1) goes into the
//    wave's region and the loads of block r+2's halo are issued.  With many
//    channels the registers do not allow that; block r+1's halo is then
//    loaded during block r's FFN, a few 16-byte pieces per lane per chunk.
//    Pixels outside the image are stored as zeros.
#pragma once
#include "cf_device.h"
#include "cf_fused_impl.h"
#include "cf_kernels.h"

namespace cf {
namespace gblk {

constexpr int GW = 8;               // group width of the grouped conv
constexpr int BR = 4, BC = 16;      // block: 4 rows x 16 columns
constexpr int HR = BR + 2, HC = BC + 2;
constexpr int HPIX = HR * HC;       // halo pixels of a block (3 x 3 taps)
constexpr int HSTEP = 4;            // halo pieces per lane per FFN chunk (many channels)

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
    int RB, SEG;                    // row bands ceil(H/4), 16-column segments ceil(W/16)
    int nblocks;                    // N * RB * SEG
    int rbase, rextra;              // rounds (NW blocks) per workgroup: rbase, +1 for the first rextra
    int xcd_map;                    // 1: workgroup i takes range (i % 8) * (G / 8) + i / 8
    uint32_t off_halo;              // LDS offset of the halo regions (after the weights)
    // the network stem in front of the block (STEM kernels): x is then the
    // stem output, computed per halo from the image and never stored
    const uint16_t *xs;             // image [N][Hin][Win][3]
    const uint16_t *sw;             // stem taps [C][3][3][3]
    const float *ss, *sb;           // stem scale, bias (NULL: 1, 0)
    int Hin, Win;
    uint32_t off_stage;             // LDS offset of the waves' image windows (STEM)
};

__device__ __forceinline__ u32x4 lds16(const uint8_t *base, uint32_t off) {
    return *reinterpret_cast<const u32x4 *>(base + off);
}
__device__ __forceinline__ void sts16(uint8_t *base, uint32_t off, const u32x4 &v) {
    *reinterpret_cast<u32x4 *>(base + off) = v;
}

// The image window a block's halo needs: rows 2 r0 - 3 .. 2 r0 + 9, columns
// 2 c0 - 3 .. 2 c0 + 33 (13 x 37 pixels), staged in LDS as 4 values a pixel
// (the 3 channels and a zero) with a 38th, zero pixel closing each row.  The
// fused kernel orders the stem's K for that layout: slot (tap row kh, tap
// column pair kw0 = 0 or 2, channel 0..3) -- 6 slices of 8, K = 64 in two
// products -- so a B fragment is one 16-byte read of two staged pixels (the
// slots of tap column 3 and channel 3 have zero weights).
constexpr int SWR = 2 * HR + 1, SWP = 2 * HC + 1;       // 13 rows, 37 pixels
constexpr int SWPIX = SWR * SWP;                         // 481
constexpr int SWL = (SWPIX + 63) / 64;                   // window pixels per lane
constexpr int SPITCH = (SWP + 1) * 8;                    // 304 bytes a staged row (a multiple of 16)
constexpr int STG = 4096;                                // LDS bytes of a wave's window (>= SWR SPITCH)

// A fragment of output channel o (taps [o][3][3][3]) for product m, K slice q
// of the staged-pixel order above (the stem kernel alone uses the same order,
// so both round the stem output alike).
__device__ __forceinline__ u32x4 stem_afrag_px(const uint16_t *sw, int o, int m, int q) {
    const int sl = 4 * m + q;
    uint32_t e[8] = {0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u};
    if (sl < 6) {
        const int kh = sl >> 1, kw0 = 2 * (sl & 1);
#pragma unroll
        for (int j = 0; j < 8; j++) {
            const int kw = kw0 + j / 4, ci = j % 4;
            if (ci < 3 && kw < 3)
                e[j] = sw[(size_t)o * 27 + (kh * 3 + kw) * 3 + ci];
        }
    }
    return u32x4{e[0] | (e[1] << 16), e[2] | (e[3] << 16), e[4] | (e[5] << 16), e[6] | (e[7] << 16)};
}

// A fragment of output channel o (taps [o][3][3][3]) for K slice q.
__device__ __forceinline__ u32x4 stem_afrag(const uint16_t *sw, int o, int q) {
    const uint16_t *wo = sw + (size_t)o * 27;
    uint32_t e[8] = {0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u};
    if (q < 3) {
#pragma unroll
        for (int j = 0; j < 8; j++)
            e[j] = wo[9 * q + j];
    } else {
        e[0] = wo[8];
        e[1] = wo[17];
        e[2] = wo[26];
    }
    return u32x4{e[0] | (e[1] << 16), e[2] | (e[3] << 16), e[4] | (e[5] << 16), e[6] | (e[7] << 16)};
}

// The B fragment of output pixel (sr, sc) for product m, K slice q of that
// order, gathered from the image (zero outside it); the stem kernel alone.
__device__ __forceinline__ u32x4 stem_bfrag_px(const uint16_t *img, int Hin, int Win, int sr, int sc, int m, int q,
                                              bool in) {
    const int sl = 4 * m + q;
    uint32_t e[8] = {0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u};
    if (in && sl < 6) {
        const int ir = 2 * sr - 1 + (sl >> 1);
        if (ir >= 0 && ir < Hin) {
#pragma unroll
            for (int pp = 0; pp < 2; pp++) {
                const int ic = 2 * sc - 1 + 2 * (sl & 1) + pp;
                if (ic >= 0 && ic < Win) {
#pragma unroll
                    for (int ci = 0; ci < 3; ci++)
                        e[4 * pp + ci] = img[((size_t)ir * Win + ic) * 3 + ci];
                }
            }
        }
    }
    return u32x4{e[0] | (e[1] << 16), e[2] | (e[3] << 16), e[4] | (e[5] << 16), e[6] | (e[7] << 16)};
}

template <int C>
struct Geo {
    static_assert(C % 16 == 0 && C >= 16, "C must be a multiple of 16");
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
    static constexpr int OFF_VEC = 3 * GROW;       // s0, b0, s2, b2: C floats each
    static constexpr int OFF_W = (OFF_VEC + 16 * C + 255) & ~255;
    static constexpr int HPIECES = HPIX * C8;      // 16-byte pieces of a halo
    static constexpr int HPL = (HPIECES + 63) / 64;
    static constexpr int HSTEPS = (HPIECES + 64 * HSTEP - 1) / (64 * HSTEP);
    static constexpr int CPIECES = (2 * KST + MO) * 64 + 16;
    // a whole block's halo in registers (one block ahead) while it is cheap
    static constexpr bool PREF2 = HPL <= 9;
};

// waves per workgroup for a channel count: 8 where their halo regions fit
constexpr int nw_for(int C) { return C <= 64 ? 8 : 4; }

// LDS bytes of a configuration: resident weights (nch chunks) or the ring
template <int C>
inline size_t lds_bytes(int nch, bool resident) {
    using G = Geo<C>;
    return (size_t)G::OFF_W + (size_t)(resident ? nch : 2) * G::CHB + (size_t)nw_for(C) * G::HALO;
}

template <int C, int NW, typename T, int ACT, bool RES, bool STEM = false>
struct GB {
    using G = Geo<C>;
    static constexpr int NT = NW * 64;
    static constexpr int PB = G::PB, C8 = G::C8, NG = G::NG, KST = G::KST, MO = G::MO, HALO = G::HALO;
    static constexpr int W1B = G::W1B, W2B = G::W2B, CHB = G::CHB, GROW = G::GROW;
    static constexpr int HPIECES = G::HPIECES, HPL = G::HPL, HSTEPS = G::HSTEPS, CPIECES = G::CPIECES;
    static constexpr bool PREF2 = G::PREF2;
    static constexpr int CPT = (CPIECES + NT - 1) / NT;
    static constexpr int STT = (HPIX + 15) / 16;  // stem: 16-pixel MFMA tiles of a halo
    static constexpr int SMT = C / 16;            // stem: 16-channel output tiles
    static constexpr int HVN = STEM ? 1 : (PREF2 ? HPL : 1);
    static_assert(!STEM || PREF2, "the stem path prefetches one block ahead");
    // ReLU and identity: s1 is folded into the staged W1 rows and b1 starts
    // the expand accumulators, so the activation is a packed convert (and a
    // packed max); GELU applies s1, b1 and erf in fp32
    static constexpr bool FOLD = ACT != ACT_GELU;

    // ---- 16-byte piece p of a chunk of the FFN weights, in fragment order.
    // Where a piece comes from does not depend on the chunk except through a
    // chunk offset, so each thread sets its pieces up once (PieceRef) and a
    // chunk load is an add and a compare per piece.
    struct PieceRef {
        int kind;      // 0 W1, 1 W2, 2 s1 / b1, 3 none
        int rowc;      // W1: row within the chunk; W2: hidden column within the chunk; 2: hidden within the chunk
        int off;       // element offset at chunk 0 (W1: row * C + col; W2: o * EC + col; 2: hidden)
        int sel;       // W1: col < C; 2: 0 = s1, 1 = b1
    };
    static __device__ __forceinline__ PieceRef piece_ref(const Args &a, int p) {
        PieceRef r{3, 0, 0, 0};
        if (p < 2 * KST * 64) {
            const int f = p >> 6, ln = p & 63, t = f / KST, kk = f - t * KST;
            const int m = ln & 15, qq = ln >> 4;
            const int row = 8 * (m >> 2) + 4 * t + (m & 3);
            const int col = 32 * kk + 8 * qq;
            r = PieceRef{0, row, row * C + col, col < C ? 1 : 0};
        } else if (p < (2 * KST + MO) * 64) {
            const int pp = p - 2 * KST * 64;
            const int mo = pp >> 6, ln = pp & 63;
            const int o = 16 * mo + (ln & 15), hc = 8 * (ln >> 4);
            r = PieceRef{1, hc, o * a.EC + hc, 0};
        } else if (p < CPIECES) {
            const int jv = p - (2 * KST + MO) * 64;  // 0..7: s1, 8..15: b1
            r = PieceRef{2, 4 * (jv & 7), 4 * (jv & 7), jv >> 3};
        }
        return r;
    }
    static __device__ __forceinline__ u32x4 piece_at(const Args &a, const PieceRef &r, int ch) {
        u32x4 v = {0u, 0u, 0u, 0u};
        const int h0 = ch * 32;
        if (r.kind == 0) {
            if (r.sel && h0 + r.rowc < a.EC) {
                v = *reinterpret_cast<const u32x4 *>(a.w1 + (size_t)h0 * C + r.off);
                if (FOLD && a.s1)
                    v = fused::scale8<T>(v, a.s1[h0 + r.rowc]);
            }
        } else if (r.kind == 1) {
            if (h0 + r.rowc < a.EC)
                v = *reinterpret_cast<const u32x4 *>(a.w2 + r.off + h0);
        } else if (r.kind == 2) {
            float4v f = {0.f, 0.f, 0.f, 0.f};
            if (h0 + r.rowc < a.EC) {
                const float *src = r.sel ? a.b1 : a.s1;
                if (src)
                    f = *reinterpret_cast<const float4v *>(src + h0 + r.off);
                else if (!r.sel)
                    f = float4v{1.f, 1.f, 1.f, 1.f};
            }
            v = __builtin_bit_cast(u32x4, f);
        }
        return v;
    }
    static __device__ __forceinline__ void chunk_load(const Args &a, const PieceRef (&pr)[CPT], int ch,
                                                      u32x4 (&r)[CPT]) {
#pragma unroll
        for (int u = 0; u < CPT; u++)
            r[u] = piece_at(a, pr[u], ch);
    }
    static __device__ __forceinline__ void chunk_store(uint8_t *slot, int tid, const u32x4 (&r)[CPT]) {
#pragma unroll
        for (int u = 0; u < CPT; u++) {
            const int p = u * NT + tid;
            if (p < CPIECES)
                sts16(slot, (uint32_t)p * 16, r[u]);
        }
    }

    // ---- block geometry (wave-uniform: scalar registers)
    struct Blk {
        int n, r0, c0;  // image, first row, first column
        bool valid;
    };
    static __device__ __forceinline__ Blk decode(const Args &a, int b) {
        Blk k;
        k.valid = b < a.nblocks;
        const int bb = k.valid ? b : 0;
        const int seg = bb % a.SEG, t = bb / a.SEG;
        const int rb = t % a.RB;
        k.n = t / a.RB;
        k.r0 = BR * rb;
        k.c0 = BC * seg;
        return k;
    }

    // halo of block k: pieces are (pixel px = r * HC + cc of the 6 x 18
    // window, 16-byte channel piece cq); the window's top-left pixel
    // (r0 - 1, c0 - 1) is the base, so a piece is a 32-bit offset from it
    struct HaloCtx {
        const uint16_t *base;  // element address of window pixel (0, 0) (may lie outside x; read only in bounds)
        int rlo, rhi, clo, chi;  // window rows r with rlo <= r < rhi and columns likewise lie in the image
        int WC;                  // W * C
    };
    static __device__ __forceinline__ HaloCtx halo_ctx(const Args &a, const Blk &k) {
        HaloCtx h;
        const int64_t pix0 = ((int64_t)k.n * a.H + (k.r0 - 1)) * a.W + (k.c0 - 1);
        h.base = a.x + pix0 * C;
        h.rlo = k.valid ? 1 - k.r0 : HR;   // an invalid block reads nothing
        h.rhi = a.H - k.r0 + 1;
        h.clo = 1 - k.c0;
        h.chi = a.W - k.c0 + 1;
        h.WC = a.W * C;
        return h;
    }
    static __device__ __forceinline__ u32x4 halo_piece(const HaloCtx &h, int i) {
        const int px = i / C8, cq = i - px * C8;
        const int r = px / HC, cc = px - r * HC;
        u32x4 v = {0u, 0u, 0u, 0u};
        if (r >= h.rlo && r < h.rhi && cc >= h.clo && cc < h.chi)
            v = *reinterpret_cast<const u32x4 *>(h.base + (r * h.WC + cc * C + 8 * cq));
        return v;
    }
    // the lane's pieces (first + u) * 64 + lane, u < NP
    template <int NP>
    static __device__ __forceinline__ void halo_load(const HaloCtx &h, int first, int lane, u32x4 (&v)[NP]) {
#pragma unroll
        for (int u = 0; u < NP; u++) {
            const int i = (first + u) * 64 + lane;
            v[u] = u32x4{0u, 0u, 0u, 0u};
            if (i < HPIECES)
                v[u] = halo_piece(h, i);
        }
    }
    // piece i lands at pixel i / C8, channel piece i % C8 of the wave's region
    template <int NP>
    static __device__ __forceinline__ void halo_store(uint8_t *reg, int first, int lane, const u32x4 (&v)[NP]) {
#pragma unroll
        for (int u = 0; u < NP; u++) {
            const int i = (first + u) * 64 + lane;
            if (i < HPIECES) {
                const int px = i / C8, cq = i - px * C8;
                sts16(reg, (uint32_t)px * PB + (uint32_t)cq * 16, v[u]);
            }
        }
    }

    // ---- the stem (STEM kernels).  The halo of a block is computed from the
    // image instead of read: halo pixel px of the 6 x 18 window is stem output
    // (sr, sc) = (r0 - 1 + px / 18, c0 - 1 + px % 18), one B column of the
    // stem products (the staged-pixel K order).  The image window is read one
    // block ahead into registers and staged in the wave's LDS window when the
    // halo is due.
    // the lane's pixels i = 64 u + lane of block k's image window, read as
    // they lie in memory: v[u] the aligned 32-bit word holding two of the
    // pixel's three values, h[u] the third one.  Bit u of m says the pixel
    // lies in the image (else pixel 0 of the image is read in its place), bit
    // 8 + u that its first element index is odd (the word then holds channels
    // 1, 2).  Nothing here waits for the loads (no branch, no use of a loaded
    // value): stem_store puts the values together a block later
    static __device__ __forceinline__ void stem_load(const Args &a, const Blk &k, int lane, uint32_t (&v)[SWL],
                                                     uint16_t (&h)[SWL], uint32_t &m) {
        const uint16_t *img = a.xs + (size_t)k.n * a.Hin * a.Win * 3;
        const int row0 = 2 * k.r0 - 3, col0 = 2 * k.c0 - 3;
        const int par0 = k.n & a.Hin & a.Win & 1;  // parity of the image's first element index
        m = 0u;
#pragma unroll
        for (int u = 0; u < SWL; u++) {
            const int i = u * 64 + lane;
            const int rr = i / SWP, pc = i - rr * SWP;
            const int ir = row0 + rr, ic = col0 + pc;
            const bool in = k.valid & (i < SWPIX) & ((unsigned)ir < (unsigned)a.Hin) & ((unsigned)ic < (unsigned)a.Win);
            const int pix = in ? ir * a.Win + ic : 0;
            const int odd = (par0 ^ pix) & 1;
            const uint16_t *e = img + (size_t)pix * 3;
            v[u] = *reinterpret_cast<const uint32_t *>(e + odd);
            h[u] = e[2 - 2 * odd];
            m |= (in ? 1u : 0u) << u | (uint32_t)odd << (8 + u);
        }
    }
    // stages block k's window (this wave only: its LDS operations run in
    // order), runs the two products of each 16-pixel halo tile from it,
    // applies s, b and ReLU, zeroes pixels outside the stem output (the
    // block's padding) and writes the halo region as the block's loads would
    // have
    static __device__ __forceinline__ void stem_store(uint8_t *reg, uint8_t *stage, const Args &a, const Blk &k,
                                                      int lane, const uint32_t (&v)[SWL], const uint16_t (&h)[SWL], uint32_t m,
                                                      const u32x4 (&sa)[SMT][2], const float4v (&ssv)[SMT],
                                                      const float4v (&sbv)[SMT]) {
        const int q = lane >> 4, jl = lane & 15;
#pragma unroll
        for (int u = 0; u < SWL; u++) {
            const int i = u * 64 + lane;
            const int rr = i / SWP, pc = i - rr * SWP;
            // channels 0, 1 | channel 2, zero; zero outside the image
            const bool in = (m >> u) & 1u, odd = (m >> (8 + u)) & 1u;
            const uint32_t w0 = odd ? ((uint32_t)h[u] | (v[u] << 16)) : v[u];
            const uint32_t w1 = odd ? (v[u] >> 16) : (uint32_t)h[u];
            if (i < SWPIX)
                *reinterpret_cast<u32x2 *>(stage + (uint32_t)rr * SPITCH + (uint32_t)pc * 8) =
                    u32x2{in ? w0 : 0u, in ? w1 : 0u};
        }
        // every tile's B fragments first, so the reads overlap the products
        u32x4 bv[STT][2];
#pragma unroll
        for (int t = 0; t < STT; t++) {
            const int px = 16 * t + jl;
            const int hr = px / HC, hc = px - hr * HC;
#pragma unroll
            for (int m = 0; m < 2; m++) {
                const int sl = 4 * m + q;  // slot slice: tap row sl / 2, tap columns 2 (sl % 2) and +1
                bv[t][m] = (sl < 6 && px < HPIX)
                               ? *reinterpret_cast<const u32x4 *>(stage + (uint32_t)(2 * hr + (sl >> 1)) * SPITCH +
                                                                  (uint32_t)(2 * hc + 2 * (sl & 1)) * 8)
                               : u32x4{0u, 0u, 0u, 0u};
            }
        }
#pragma unroll
        for (int t = 0; t < STT; t++) {
            const int px = 16 * t + jl;
            const int hr = px / HC, hc = px - hr * HC;
            const int sr = k.r0 - 1 + hr, sc = k.c0 - 1 + hc;
            const bool in = k.valid & (px < HPIX) & ((unsigned)sr < (unsigned)a.H) & ((unsigned)sc < (unsigned)a.W);
#pragma unroll
            for (int mt = 0; mt < SMT; mt++) {
                float4v acc = T::mfma(sa[mt][0], bv[t][0], float4v{0.f, 0.f, 0.f, 0.f});
                acc = T::mfma(sa[mt][1], bv[t][1], acc);
                float uu[4];
#pragma unroll
                for (int e4 = 0; e4 < 4; e4++)
                    uu[e4] = in ? fmaxf(fmaf(acc[e4], ssv[mt][e4], sbv[mt][e4]), 0.0f) : 0.0f;
                if (px < HPIX)
                    *reinterpret_cast<u32x2 *>(reg + (uint32_t)px * PB + (uint32_t)(16 * mt + 4 * q) * 2) =
                        u32x2{T::pack2(uu[0], uu[1]), T::pack2(uu[2], uu[3])};
            }
        }
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
        const int tid = threadIdx.x, lane = tid & 63;
        const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform: block indices stay scalar
        const int q = lane >> 4, jl = lane & 15;
        const int Gn = gridDim.x;
        const int gi = a.xcd_map ? (int)(blockIdx.x % 8) * (Gn / 8) + (int)(blockIdx.x / 8) : (int)blockIdx.x;
        const int nr = a.rbase + (gi < a.rextra ? 1 : 0);
        const int rstart = gi * a.rbase + (gi < a.rextra ? gi : a.rextra);
        if (nr == 0)
            return;  // uniform over the workgroup, before any barrier

        uint8_t *gwl = smem;
        uint8_t *wts = smem + G::OFF_W;
        uint8_t *reg = smem + a.off_halo + wv * HALO;
        const float *vec = reinterpret_cast<const float *>(smem + G::OFF_VEC);

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
            reinterpret_cast<float *>(smem + G::OFF_VEC)[i] = src ? src[c] : (v == 0 || v == 2 ? 1.0f : 0.0f);
        }
        // FFN weights: every chunk (resident), or chunk 0 in slot 0 with chunk
        // 1 waiting in registers (ring)
        u32x4 cA[CPT], cB[CPT];
        PieceRef pref[CPT];
#pragma unroll
        for (int u = 0; u < CPT; u++)
            pref[u] = piece_ref(a, u * NT + tid);
        if constexpr (RES) {
            for (int ch = 0; ch < a.nch; ch++) {
                chunk_load(a, pref, ch, cA);
                chunk_store(wts + (uint32_t)ch * CHB, tid, cA);
            }
        } else {
            chunk_load(a, pref, 0, cA);
            chunk_store(wts, tid, cA);
            chunk_load(a, pref, a.nch > 1 ? 1 : 0, cA);
        }
        // stem (STEM kernels): the lane's A fragments (output channel 16 mt +
        // jl, K slice q as in stem_load) and the scale/bias of its D rows
        u32x4 sa[STEM ? SMT : 1][2];
        float4v ssv[STEM ? SMT : 1], sbv[STEM ? SMT : 1];
        if constexpr (STEM) {
            // the wave's window: its pad slots (the 38th pixel of a row) stay zero
            for (int i = lane; i < STG / 16; i += 64)
                *reinterpret_cast<u32x4 *>(smem + a.off_stage + wv * STG + i * 16) = u32x4{0u, 0u, 0u, 0u};
#pragma unroll
            for (int mt = 0; mt < SMT; mt++) {
                sa[mt][0] = stem_afrag_px(a.sw, 16 * mt + jl, 0, q);
                sa[mt][1] = stem_afrag_px(a.sw, 16 * mt + jl, 1, q);
#pragma unroll
                for (int e4 = 0; e4 < 4; e4++) {
                    const int c = 16 * mt + 4 * q + e4;
                    ssv[mt][e4] = a.ss ? a.ss[c] : 1.0f;
                    sbv[mt][e4] = a.sb ? a.sb[c] : 0.0f;
                }
            }
        }
        // halo of the first block; with PREF2 the second block's waits in registers
        u32x4 hv[HVN];
        uint32_t hs[STEM ? SWL : 1], hm = 0u;
        uint16_t hh[STEM ? SWL : 1];
        uint8_t *stage = smem + a.off_stage + wv * STG;
        if constexpr (STEM) {
            const Blk k0 = decode(a, rstart * NW + wv);
            stem_load(a, k0, lane, hs, hh, hm);
            stem_store(reg, stage, a, k0, lane, hs, hh, hm, sa, ssv, sbv);
            if (nr > 1)
                stem_load(a, decode(a, (rstart + 1) * NW + wv), lane, hs, hh, hm);
        } else {
            const HaloCtx h0 = halo_ctx(a, decode(a, rstart * NW + wv));
            for (int s = 0; s < HSTEPS; s++) {
                u32x4 v[HSTEP];
                halo_load<HSTEP>(h0, s * HSTEP, lane, v);
                halo_store<HSTEP>(reg, s * HSTEP, lane, v);
            }
            if constexpr (PREF2) {
                if (nr > 1)
                    halo_load<HPL>(halo_ctx(a, decode(a, (rstart + 1) * NW + wv)), 0, lane, hv);
            }
        }
        __syncthreads();

        // per-lane conv constants: A operand row (s, o) and tap row i = q - s
        const int cs = jl >> 3, co = jl & 7;
        const int ti = q - cs;
        const bool tap_ok = ti >= 0 && ti <= 2;
        const uint32_t a_off = (uint32_t)(tap_ok ? ti : 0) * GROW + (uint32_t)co * 16;
        // D rows of this lane: block row 2p + (q >> 1), channels 8g + 4 (q & 1) + e
        const int drow = q >> 1, dch = 4 * (q & 1);

        // block state
        u32x4 dfr[BR][KST];
        float4v acc[BR][MO];
        u32x2 xres[BR][MO];  // the block input at the lane's output elements (residual)
        Blk kcur;
        int cur_r = 0;

        // ---- start of block r: conv, d, B fragments, halo prefetch
        auto block_begin = [&](int r) {
            cur_r = r;
            kcur = decode(a, (rstart + r) * NW + wv);
            // the residual comes from the halo (centre pixels), read before the
            // conv outputs overwrite the region; no global re-read in the epilogue
#pragma unroll
            for (int nt = 0; nt < BR; nt++)
#pragma unroll
                for (int mo = 0; mo < MO; mo++)
                    xres[nt][mo] = *reinterpret_cast<const u32x2 *>(
                        reg + (uint32_t)((nt + 1) * HC + jl + 1) * PB + (uint32_t)(16 * mo + 4 * q) * 2);
#pragma unroll
            for (int g = 0; g < NG; g++) {
                const int c = GW * g + dch;
                const float4v sc = *reinterpret_cast<const float4v *>(vec + c);
                const float4v bi = *reinterpret_cast<const float4v *>(vec + C + c);
                u32x4 av[3];
#pragma unroll
                for (int dj = 0; dj < 3; dj++)
                    av[dj] = tap_ok ? lds16(gwl, a_off + (uint32_t)(dj * C + GW * g) * 16) : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
                for (int pr = 0; pr < BR / 2; pr++) {
                    float4v cacc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int dj = 0; dj < 3; dj++) {
                        const u32x4 bv =
                            lds16(reg, (uint32_t)((2 * pr + q) * HC + jl + dj) * PB + (uint32_t)g * 16);
                        cacc = T::mfma(av[dj], bv, cacc);
                    }
                    float v[4];
#pragma unroll
                    for (int e = 0; e < 4; e++)
                        v[e] = fmaf(cacc[e], sc[e], bi[e]);
                    *reinterpret_cast<u32x2 *>(reg + (uint32_t)((2 * pr + drow) * BC + jl) * PB + (uint32_t)c * 2) =
                        u32x2{T::pack2(v[0], v[1]), T::pack2(v[2], v[3])};
                }
            }
#pragma unroll
            for (int nt = 0; nt < BR; nt++)
#pragma unroll
                for (int kk = 0; kk < KST; kk++)
                    dfr[nt][kk] = (32 * kk + 8 * q < C)
                                      ? lds16(reg, (uint32_t)(nt * BC + jl) * PB + (uint32_t)(32 * kk + 8 * q) * 2)
                                      : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
            for (int nt = 0; nt < BR; nt++)
#pragma unroll
                for (int mo = 0; mo < MO; mo++)
                    acc[nt][mo] = float4v{0.f, 0.f, 0.f, 0.f};
            if constexpr (STEM) {
                // the region is free: block r+1's stem output in, block r+2's
                // image fragments out
                if (r + 1 < nr)
                    stem_store(reg, stage, a, decode(a, (rstart + r + 1) * NW + wv), lane, hs, hh, hm, sa, ssv, sbv);
                if (r + 2 < nr)
                    stem_load(a, decode(a, (rstart + r + 2) * NW + wv), lane, hs, hh, hm);
            } else if constexpr (PREF2) {
                // the region is free: block r+1's halo in, block r+2's loads out
                if (r + 1 < nr)
                    halo_store<HPL>(reg, 0, lane, hv);
                if (r + 2 < nr)
                    halo_load<HPL>(halo_ctx(a, decode(a, (rstart + r + 2) * NW + wv)), 0, lane, hv);
            }
        };

        // ---- one hidden chunk of the current block from weights at `cw`
        auto chunk = [&](int ch, const uint8_t *cw) {
            u32x4 sv[HSTEP];
            const bool hstep = !PREF2 && cur_r + 1 < nr && ch < HSTEPS;
            if (hstep)
                halo_load<HSTEP>(halo_ctx(a, decode(a, (rstart + cur_r + 1) * NW + wv)), ch * HSTEP, lane, sv);
            float s1v[8], b1v[8];
            {
                const float4v s_lo = *reinterpret_cast<const float4v *>(cw + W1B + W2B + 32 * q);
                const float4v s_hi = *reinterpret_cast<const float4v *>(cw + W1B + W2B + 32 * q + 16);
                const float4v b_lo = *reinterpret_cast<const float4v *>(cw + W1B + W2B + 128 + 32 * q);
                const float4v b_hi = *reinterpret_cast<const float4v *>(cw + W1B + W2B + 128 + 32 * q + 16);
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
                    a1[t][kk] = lds16(cw, (uint32_t)(t * KST + kk) * 1024 + (uint32_t)lane * 16);
            u32x4 gfr[BR];
#pragma unroll
            for (int nt = 0; nt < BR; nt++) {
                float u[8];
#pragma unroll
                for (int t = 0; t < 2; t++) {
                    float4v e = FOLD ? float4v{b1v[4 * t], b1v[4 * t + 1], b1v[4 * t + 2], b1v[4 * t + 3]}
                                     : float4v{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int kk = 0; kk < KST; kk++)
                        e = T::mfma(a1[t][kk], dfr[nt][kk], e);
#pragma unroll
                    for (int i = 0; i < 4; i++)
                        u[4 * t + i] = FOLD ? e[i] : act(fmaf(e[i], s1v[4 * t + i], b1v[4 * t + i]));
                }
                if constexpr (FOLD && ACT == ACT_RELU && !T::is_bf16) {
                    // round, then the packed max: max(round(u), 0) = round(max(u, 0))
                    u32x4 g;
#pragma unroll
                    for (int i = 0; i < 4; i++)
                        g[i] = __builtin_bit_cast(
                            uint32_t, __builtin_elementwise_max(__builtin_bit_cast(half2v, T::pack2(u[2 * i], u[2 * i + 1])),
                                                                half2v{(_Float16)0.0f, (_Float16)0.0f}));
                    gfr[nt] = g;
                } else {
                    if constexpr (FOLD && ACT == ACT_RELU)
#pragma unroll
                        for (int i = 0; i < 8; i++)
                            u[i] = fmaxf(u[i], 0.0f);
                    gfr[nt] = u32x4{T::pack2(u[0], u[1]), T::pack2(u[2], u[3]), T::pack2(u[4], u[5]),
                                    T::pack2(u[6], u[7])};
                }
            }
#pragma unroll
            for (int mo = 0; mo < MO; mo++) {
                const u32x4 a2 = lds16(cw, (uint32_t)W1B + (uint32_t)mo * 1024 + (uint32_t)lane * 16);
#pragma unroll
                for (int nt = 0; nt < BR; nt++)
                    acc[nt][mo] = T::mfma(a2, gfr[nt], acc[nt][mo]);
            }
            if (hstep)
                halo_store<HSTEP>(reg, ch * HSTEP, lane, sv);
        };

        // ---- end of block: remaining halo steps, epilogue y = x + s2 acc + b2
        auto block_end = [&]() {
            if constexpr (!PREF2) {
                if (cur_r + 1 < nr) {
                    const HaloCtx hn = halo_ctx(a, decode(a, (rstart + cur_r + 1) * NW + wv));
                    for (int s = a.nch; s < HSTEPS; s++) {
                        u32x4 v[HSTEP];
                        halo_load<HSTEP>(hn, s * HSTEP, lane, v);
                        halo_store<HSTEP>(reg, s * HSTEP, lane, v);
                    }
                }
            }
            if (!kcur.valid)
                return;
#pragma unroll
            for (int nt = 0; nt < BR; nt++) {
                const int h = kcur.r0 + nt, w = kcur.c0 + jl;
                if (h >= a.H || w >= a.W)
                    continue;
                const size_t pix = ((size_t)kcur.n * a.H + h) * a.W + w;
#pragma unroll
                for (int mo = 0; mo < MO; mo++) {
                    const int c = 16 * mo + 4 * q;
                    const u32x2 xv = xres[nt][mo];
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
        };

        if constexpr (RES) {
            // every chunk resident: the waves run independently from here on
            for (int r = 0; r < nr; r++) {
                block_begin(r);
                for (int ch = 0; ch < a.nch; ch++)
                    chunk(ch, wts + (uint32_t)ch * CHB);
                block_end();
            }
        } else {
            // ring: global chunk step j = r * nch + ch uses slot j & 1.  On
            // entry to step j the slot holds chunk j and the register set
            // `pend` holds chunk j+1; the step loads chunk j+2 into the other
            // set, computes chunk j, stores `pend` into the other slot and
            // passes the barrier.  Steps go in pairs so that each register
            // set keeps a fixed role.
            const int total = nr * a.nch;
            auto step = [&](int j, u32x4 (&pend)[CPT], u32x4 (&next)[CPT]) {
                const int r = j / a.nch, ch = j - r * a.nch;
                if (ch == 0)
                    block_begin(r);
                chunk_load(a, pref, (j + 2) % a.nch, next);  // (past the last step: unused reloads)
                chunk(ch, wts + (uint32_t)(j & 1) * CHB);
                chunk_store(wts + (uint32_t)((j + 1) & 1) * CHB, tid, pend);
                __syncthreads();
                if (ch == a.nch - 1)
                    block_end();
            };
            for (int j = 0; j < total; j += 2) {
                step(j, cA, cB);
                if (j + 1 < total)
                    step(j + 1, cB, cA);
            }
        }
    }
};

template <int C, int NW, typename T, int ACT, bool RES, bool STEM = false>
__global__ __launch_bounds__(NW * 64, 1) void gblock_kernel(Args a) {
    extern __shared__ __attribute__((aligned(256))) uint8_t smem[];
    GB<C, NW, T, ACT, RES, STEM>::run(a, smem);
}

// The grouped block on x, or (STEM) the stem and the block on the image
// stem->x; s describes the block (its H, W are the stem output's).
template <int C, bool STEM = false>
hipError_t launch_c(const void *x, void *y, const GBlockW &w, const Shape &s, hipStream_t st,
                    const StemW *stem = nullptr) {
    constexpr int NW = nw_for(C);
    Args a{};
    if constexpr (STEM) {
        a.xs = (const uint16_t *)stem->x;
        a.sw = (const uint16_t *)stem->w;
        a.ss = stem->s;
        a.sb = stem->b;
        a.Hin = stem->Hin;
        a.Win = stem->Win;
    }
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
    a.RB = (s.H + BR - 1) / BR;
    a.SEG = (s.W + BC - 1) / BC;
    const int64_t nb = (int64_t)s.N * a.RB * a.SEG;
    if (nb > ((int64_t)1 << 30))
        return hipErrorInvalidValue;
    a.nblocks = (int)nb;
    const int rounds = (int)((nb + NW - 1) / NW);
    const int cus = device_cu_count();
    const int Gn = rounds < cus ? rounds : cus;
    a.rbase = rounds / Gn;
    a.rextra = rounds % Gn;
    a.xcd_map = (Gn % 8 == 0) ? 1 : 0;
    const size_t stg = STEM ? (size_t)NW * STG : 0;  // the waves' image windows, after the halos
    const size_t lds_res = lds_bytes<C>(a.nch, true) + stg;
    const bool res = lds_res <= 160 * 1024;
    const size_t lds = res ? lds_res : lds_bytes<C>(a.nch, false) + stg;
    if (lds > 160 * 1024)
        return hipErrorInvalidConfiguration;
    a.off_stage = (uint32_t)(lds - stg);
    a.off_halo = (uint32_t)(lds - stg - (size_t)NW * Geo<C>::HALO);
    hipError_t e;
#define CF_GB_LAUNCH(TT, AC)                                                                          \
    {                                                                                                 \
        auto kf = res ? gblock_kernel<C, NW, TT, AC, true, STEM> : gblock_kernel<C, NW, TT, AC, false, STEM>; \
        if ((e = allow_full_lds((const void *)kf)) != hipSuccess)                                     \
            return e;                                                                                 \
        hipLaunchKernelGGL(kf, dim3(Gn), dim3(NW * 64), lds, st, a);                                  \
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
