// cf_cfs2.hip -- the stride-2 ConvFirst block (Fig. f:convfirst-block (c))
// in one kernel: grouped 3 x 3 conv (group width 8) C -> C with its folded
// norm at the input size, BlurPool (Triangle-3 taps [1, 2, 1] / 4 per
// direction, one pixel of reflect padding, stride 2) of the conv output and
// of the block input, the two maps concatenated (2C channels, conv output
// first) into the expand, activation, project to K, no residual.
//
// Work unit: 16 output pixels of one output row (columns j0 .. j0 + 15).
// The waves are persistent: each takes units blockIdx * nw + wave, then
// every gridDim * nw-th, in a private LDS region; the taps, s0, b0, s1, b1,
// s2 and b2 are staged in LDS once per workgroup.  Per unit:
//  1. the input window, rows 2i - 2 .. 2i + 2 and columns 2j0 - 2 .. 2j0 + 32,
//     zero outside the image (the conv's padding): every lane's pieces are
//     loaded with one batch of 16-byte loads (addresses clamped into the
//     image, the zeros selected at the LDS store); with up to 32 channels
//     the next unit's window is loaded during this unit's conv and FFN;
//  2. the grouped conv at full resolution, rows 2i - 1 .. 2i + 1 and columns
//     2j0 - 1 .. 2j0 + 31 (the positions the blur reads, before reflection),
//     on v_mfma_f32_16x16x32: for group g and tap column dj, A row m = 8s + o
//     at K index 8R + t is the tap W[R - s][dj][8g + o][t] (zero unless
//     0 <= R - s <= 2) and B column j at K index 8R + t is window pixel
//     (w0 + R, c + j + dj), channel 8g + t, so one product per tap column
//     gives conv rows w0 and w0 + 1 of 16 columns; two row sets (w0 = 0, and
//     w0 = 1 keeping only its second row) and three column tiles (the third
//     for column 2j0 + 31 alone) cover the 3 x 33 positions.  The A
//     fragments of a group (one per tap column) stay in registers for all
//     its products; s0, b0; rounded to the I/O dtype;
//  3. the blur of both maps (fp32, rounded to the I/O dtype), each read at
//     the reflected positions, into a 16-pixel tile of 2C channels,
//     zero-padded to a multiple of 32;
//  4. the FFN on v_mfma_f32_16x16x32 in chunks of 32 hidden channels:
//     expand tiles of 16 hidden channels (A = W1 rows, B = the tile), s1, b1
//     and the activation in fp32, rounded; two tiles form the B operand of
//     the project with the K order position 8q + e <-> hidden 32kk + 4q + e
//     (e < 4) or 32kk + 16 + 4q + e - 4, the lane layout the expand leaves,
//     and the W2 fragments are read in that order; s2, b2; y stored once.
//     When W1 and W2 fit in LDS beside the regions with two waves per
//     SIMD (or as many as without them), the workgroup stages them there
//     once (rows padded by 16 bytes, so the sixteen rows of a fragment read
//     fall in distinct banks) and the fragments are read from LDS.  Otherwise a chunk's W1 and W2
//     pieces are loaded from global memory (L2) one chunk ahead, the first
//     chunk's during the conv.  Every load of the loop is unconditional (addresses clamped; the
//     rows past R meet zero hidden values, the rows past K are not stored),
//     so the waits count exactly.  The loads are row-major -- lane 4r + p
//     takes piece p of row r, four adjacent lanes on one contiguous run --
//     and ds_bpermute from lane 4 jl + q moves each dword to the fragment
//     lane (jl, q) when the chunk is used (a fragment-order load, sixteen
//     rows in sixteen adjacent lanes, costs the memory unit several times
//     more per byte).
// The input windows of neighbouring units overlap by three columns and the
// conv positions on the unit's border columns are evaluated by both units.
// Conv positions outside the image are evaluated on the zero padding and
// never read: the blur's reflection of row -1 is row 1, of row H is H - 2,
// both inside the unit's rows (and likewise for columns).
#include "cf_device.h"
#include "cf_kernels.h"

namespace cf {
namespace cfs2 {

constexpr int XR = 5, XC = 35;  // input window: rows 2i-2 .. 2i+2, columns 2j0-2 .. 2j0+32
constexpr int VR = 3, VC = 33;  // conv outputs: rows 2i-1 .. 2i+1, columns 2j0-1 .. 2j0+31
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
    uint32_t off_w1, off_w2;  // LDS: taps, s0, b0, s1, b1, s2, b2; W1 and W2 when staged;
    uint32_t off_region;      // then one region per wave
};

__device__ __forceinline__ int clampi(int v, int lo, int hi) { return v < lo ? lo : (v > hi ? hi : v); }

// v_mul_u32_u24 (both factors below 2^24)
__device__ __forceinline__ uint32_t mul24(uint32_t a, uint32_t b) { return (uint32_t)__umul24(a, b); }

// one pixel of reflect padding (-1 -> 1, n -> n - 2); past that (the padded
// pixels of a unit at the right edge, whose outputs are not stored) the last
// column
__device__ __forceinline__ int refl(int v, int n) {
    int r = v < 0 ? -v : v;
    r = r == n ? n - 2 : r;
    return r < n ? r : n - 1;
}

__device__ __forceinline__ float act_f(float u, int act) {
    if (act == ACT_RELU)
        return fmaxf(u, 0.0f);
    if (act == ACT_GELU)
        return 0.5f * u * (1.0f + erff(u * 0.70710678118654752f));
    return u;
}

// LDS bytes of the staged taps and vectors
__host__ __device__ inline uint32_t staged_bytes(int C, int R, int K) {
    return ((uint32_t)(9 * C * 16 + 4 * (2 * C + 2 * R + 2 * K)) + 255) & ~255u;
}

// row strides of W1 and W2 staged in LDS
__host__ __device__ inline uint32_t w1_stride(int C) { return (uint32_t)(4 * C + 16); }
__host__ __device__ inline uint32_t w2_stride(int R) { return (uint32_t)(2 * R + 16); }
__host__ __device__ inline uint32_t weights_bytes(int C, int R, int K) {
    return ((uint32_t)R * w1_stride(C) + (uint32_t)K * w2_stride(R) + 255) & ~255u;
}

template <typename T, int C, int OTM, bool WL>
struct Kern {
    static constexpr int G = C / 8;                            // groups of the conv
    static constexpr uint32_t PP = 2 * C + 16;                 // LDS bytes per window / conv pixel
    static constexpr int C2 = 2 * C, C2P = (C2 + 31) / 32 * 32;
    static constexpr int KS = C2P / 32;                        // expand K steps
    static constexpr uint32_t PZ = 2 * C2P + 16;               // LDS bytes per tile pixel
    static constexpr uint32_t XB = XR * XC * PP, VB = VR * VC * PP, ZB = UPX * PZ;
    static constexpr uint32_t REGION = XB + VB + ZB;
    static constexpr int NX = XR * XC * G;                     // 16-byte pieces of a window
    static constexpr int NIT = (NX + 63) / 64;                 // per lane
    static constexpr bool PREF = G <= 4;                       // next window loaded during this unit

    struct Frag {
        u32x4 w1[2][KS];
        u32x2 w2[OTM][2];
    };

    struct Unit {
        int n, i, j0;
    };

    static __device__ __forceinline__ Unit decode(const Args &a, int u) {
        const int jt = u % a.jt, ni = u / a.jt;
        return Unit{ni / a.Ho, ni % a.Ho, jt * UPX};
    }

    // window piece it of this lane: pixel (rr, cc) of the window, 16-byte
    // piece pc; adjacent lanes on adjacent pieces
    // piece it of a lane: window pixel px = (rr, cc), 16-byte piece pc;
    // adjacent lanes on adjacent pieces; lanes past the last piece take the
    // last piece again
    struct Piece {
        int px, pc, rr, cc;
    };
    static __device__ __forceinline__ Piece piece(int lane, int it) {
        const int t = lane + 64 * it, tt = t < NX ? t : NX - 1;
        const int px = tt / G, rr = px / XC;
        return Piece{px, tt - px * G, rr, px - rr * XC};
    }

    // the piece's 16 bytes of image n at window origin (r0, c0), the
    // position clamped into the image (the pieces outside are stored as
    // zeros)
    static __device__ __forceinline__ u32x4 load_piece(const Args &a, const Unit &un, const Piece &p) {
        const int gr = clampi(2 * un.i - 2 + p.rr, 0, a.H - 1), gc = clampi(2 * un.j0 - 2 + p.cc, 0, a.W - 1);
        const uint32_t pix = mul24((uint32_t)gr, (uint32_t)a.W) + (uint32_t)gc;
        const uint16_t *xn = a.x + (size_t)un.n * a.H * a.W * C;
        return *reinterpret_cast<const u32x4 *>(xn + (size_t)pix * C + p.pc * 8);
    }

    static __device__ __forceinline__ void load_window(const Args &a, int u, int lane, u32x4 (&xv)[NIT]) {
        const Unit un = decode(a, u);
#pragma unroll
        for (int it = 0; it < NIT; it++)
            xv[it] = load_piece(a, un, piece(lane, it));
    }

    // this unit's window into LDS; with PREF the next unit's pieces are
    // loaded into the same registers as they are stored
    static __device__ __forceinline__ void store_window(const Args &a, int u, int next, int lane, u32x4 (&xv)[NIT],
                                                        uint8_t *X) {
        const Unit un = decode(a, u), nx = decode(a, next);
        const int r0 = 2 * un.i - 2, c0 = 2 * un.j0 - 2;
#pragma unroll
        for (int it = 0; it < NIT; it++) {
            const Piece p = piece(lane, it);
            const int gr = r0 + p.rr, gc = c0 + p.cc;
            const bool in = gr >= 0 && gr < a.H && gc >= 0 && gc < a.W;
            *reinterpret_cast<u32x4 *>(X + (uint32_t)p.px * PP + (uint32_t)p.pc * 16) =
                in ? xv[it] : u32x4{0u, 0u, 0u, 0u};
            if (PREF)
                xv[it] = load_piece(a, nx, p);
        }
    }

    // the W1 and W2 pieces of hidden chunk kk in row-major lane order: lane
    // 4r + p holds W1 row 32kk + 16t + r, columns 32ks + 8p .. + 7 (the
    // fragment piece of lane (r, p)), and W2 row 16 ot + r, hidden
    // 32kk + 4p .. + 3 and 32kk + 16 + 4p .. + 3.  Rows are clamped into the
    // matrices; W1 columns past 2C meet zero tile entries.
    static __device__ __forceinline__ void load_frag(const Args &a, int kk, int lr, int lp, Frag &f) {
        const int R = a.R;
#pragma unroll
        for (int t = 0; t < 2; t++) {
            const int hr = min(32 * kk + 16 * t + lr, R - 1);
            const uint16_t *wr = a.w1 + (size_t)hr * C2;
#pragma unroll
            for (int ks = 0; ks < KS; ks++) {
                const int k = 32 * ks + 8 * lp;
                f.w1[t][ks] = *reinterpret_cast<const u32x4 *>(wr + (k < C2 ? k : 0));
            }
        }
        const int ha = 32 * kk + 4 * lp, hb = ha + 16 < R ? ha + 16 : ha;
#pragma unroll
        for (int ot = 0; ot < OTM; ot++) {
            const uint16_t *wr = a.w2 + (size_t)min(16 * ot + lr, a.K - 1) * R;
            f.w2[ot][0] = *reinterpret_cast<const u32x2 *>(wr + ha);
            f.w2[ot][1] = *reinterpret_cast<const u32x2 *>(wr + hb);
        }
    }

    static __device__ __forceinline__ uint32_t perm(int idx, uint32_t v) {
        return (uint32_t)__builtin_amdgcn_ds_bpermute(idx, (int)v);
    }

    static __device__ void run(const Args &a, uint8_t *smem) {
        const int tid = threadIdx.x, lane = tid & 63;
        const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
        const int R = a.R, K = a.K;
        // the taps [3][3][C][8] and the vectors, once per workgroup
        for (int i = tid; i < 9 * C; i += a.nw * 64)
            *reinterpret_cast<u32x4 *>(smem + (uint32_t)i * 16) =
                *reinterpret_cast<const u32x4 *>(a.gw + (size_t)i * 8);
        float *s0l = reinterpret_cast<float *>(smem + 9 * C * 16), *b0l = s0l + C, *s1l = b0l + C, *b1l = s1l + R,
              *s2l = b1l + R, *b2l = s2l + K;
        for (int c = tid; c < C; c += a.nw * 64) {
            s0l[c] = a.s0 ? a.s0[c] : 1.0f;
            b0l[c] = a.b0 ? a.b0[c] : 0.0f;
        }
        for (int h = tid; h < R; h += a.nw * 64) {
            s1l[h] = a.s1 ? a.s1[h] : 1.0f;
            b1l[h] = a.b1 ? a.b1[h] : 0.0f;
        }
        for (int o = tid; o < K; o += a.nw * 64) {
            s2l[o] = a.s2 ? a.s2[o] : 1.0f;
            b2l[o] = a.b2 ? a.b2[o] : 0.0f;
        }
        if constexpr (WL) {
            // W1 [R][2C] and W2 [K][R] in 16-byte pieces, adjacent threads on
            // adjacent pieces
            for (int i = tid; i < R * (C / 4); i += a.nw * 64) {
                const int r = i / (C / 4), pc = i - r * (C / 4);
                *reinterpret_cast<u32x4 *>(smem + a.off_w1 + (uint32_t)r * w1_stride(C) + (uint32_t)pc * 16) =
                    *reinterpret_cast<const u32x4 *>(a.w1 + (size_t)i * 8);
            }
            for (int i = tid; i < K * (R / 8); i += a.nw * 64) {
                const int r = i / (R / 8), pc = i - r * (R / 8);
                *reinterpret_cast<u32x4 *>(smem + a.off_w2 + (uint32_t)r * w2_stride(R) + (uint32_t)pc * 16) =
                    *reinterpret_cast<const u32x4 *>(a.w2 + (size_t)i * 8);
            }
        }
        __syncthreads();
        int unit = (int)blockIdx.x * a.nw + wv;
        if (unit >= a.units)
            return;  // (after the workgroup's only barrier)
        const int stride = (int)gridDim.x * a.nw;
        const int H = a.H, W = a.W, NKK = (R + 31) / 32, OT = (K + 15) / 16;
        uint8_t *X = smem + a.off_region + (uint32_t)wv * REGION, *V = X + XB, *Z = V + VB;
        u32x4 xv[NIT];
        load_window(a, unit, lane, xv);
        for (;;) {
            // every lane-dependent index is recomputed from an opaque copy of
            // the lane index in every unit: hoisted out of the loop (one per
            // window piece, conv operand and weight row) they would hold
            // most of the registers for the whole kernel
            int ln = lane;
            asm volatile("" : "+v"(ln));
            const int q = ln >> 4, jl = ln & 15;
            const int lr = ln >> 2, lp = ln & 3, pidx = (4 * jl + q) * 4;  // row-major lane, its fragment source
            const Unit un = decode(a, unit);
            const int i = un.i, j0 = un.j0, r0 = 2 * i - 2, c0 = 2 * j0 - 2;
            // 1. the window into LDS; the first FFN chunk's fragments and,
            //    with few channels, the next unit's window in flight
            const int next = unit + stride;
            Frag f;
            if constexpr (!WL)
                load_frag(a, 0, lr, lp, f);
            store_window(a, unit, next < a.units ? next : unit, ln, xv, X);

            // 2. the grouped conv on the matrix unit (one group at a time:
            //    an unrolled group loop hoists the LDS reads of later groups
            //    and runs out of registers)
#pragma unroll 1
            for (int g = 0; g < G; g++) {
                // A lane (row jl = 8s + o, K 8q .. 8q + 7): tap row q - s
                const int di = q - (jl >> 3);
                const bool tap = di >= 0 && di <= 2;
                u32x4 av[3];
#pragma unroll
                for (int dj = 0; dj < 3; dj++) {
                    const u32x4 v = *reinterpret_cast<const u32x4 *>(
                        smem + (uint32_t)((((tap ? di : 0) * 3 + dj) * C + 8 * g + (jl & 7)) * 16));
                    av[dj] = tap ? v : u32x4{0u, 0u, 0u, 0u};
                }
                // D lane (column jl, rows 4q .. 4q + 3): conv row w0 + (q >> 1),
                // channels 8g + 4 (q & 1) .. + 3
                const int cd = 8 * g + 4 * (q & 1);
                float sc[4], bi[4];
#pragma unroll
                for (int e = 0; e < 4; e++) {
                    sc[e] = s0l[cd + e];
                    bi[e] = b0l[cd + e];
                }
#pragma unroll
                for (int rs = 0; rs < 2; rs++)
#pragma unroll
                    for (int ct = 0; ct < 3; ct++) {
                        const int vc = 16 * ct + jl, vcl = vc < VC ? vc : VC - 1;  // columns past 32 are not kept
                        const uint8_t *bp = X + (uint32_t)((rs + q) * XC + vcl) * PP + (uint32_t)g * 16;
                        float4v d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                        for (int dj = 0; dj < 3; dj++)
                            d = T::mfma(av[dj], *reinterpret_cast<const u32x4 *>(bp + dj * PP), d);
                        if ((rs == 0 || q >= 2) && vc < VC)
                            *reinterpret_cast<u32x2 *>(V + (uint32_t)((rs + (q >> 1)) * VC + vc) * PP +
                                                       (uint32_t)cd * 2) =
                                u32x2{T::pack2(fmaf(d[0], sc[0], bi[0]), fmaf(d[1], sc[1], bi[1])),
                                      T::pack2(fmaf(d[2], sc[2], bi[2]), fmaf(d[3], sc[3], bi[3]))};
                    }
            }

            // 3. BlurPool of the conv output and of the input (reflected
            //    positions; the conv map sits one row and one column inside
            //    the window) into the tile [16][C2P]
            //    Lane-constant per pass: the pixel, the four channels, the
            //    map they come from (its base and row stride); the rows'
            //    reflections are wave-uniform.
            const uint32_t xr0 = refl(2 * i - 1, H) - r0, xr1 = 2, xr2 = refl(2 * i + 1, H) - r0;
#pragma unroll 2
            for (int t = ln; t < UPX * (C2P / 4); t += 64) {
                const int px = t / (C2P / 4), c = 4 * (t - px * (C2P / 4));
                const bool cz = C2P == C2 || c < C2;      // zero padding past 2C
                const int cc = cz ? c : 0;
                const bool isv = cc < C;
                const uint32_t base = isv ? (uint32_t)(V - X) - (uint32_t)(VC + 1) * PP + (uint32_t)cc * 2
                                          : (uint32_t)(cc - C) * 2;
                const uint32_t rst = isv ? (uint32_t)VC * PP : (uint32_t)XC * PP;
                const uint32_t ro[3] = {mul24(xr0, rst), mul24(xr1, rst), mul24(xr2, rst)};
                uint32_t co[3];
#pragma unroll
                for (int tb = 0; tb < 3; tb++)
                    co[tb] = mul24((uint32_t)(refl(2 * (j0 + px) + tb - 1, W) - c0), PP);
                float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ta = 0; ta < 3; ta++)
#pragma unroll
                    for (int tb = 0; tb < 3; tb++) {
                        const float wt = (ta == 1 ? 0.5f : 0.25f) * (tb == 1 ? 0.5f : 0.25f);
                        const u32x2 v = *reinterpret_cast<const u32x2 *>(X + base + ro[ta] + co[tb]);
                        acc[0] = fmaf(wt, T::lo(v[0]), acc[0]);
                        acc[1] = fmaf(wt, T::hi(v[0]), acc[1]);
                        acc[2] = fmaf(wt, T::lo(v[1]), acc[2]);
                        acc[3] = fmaf(wt, T::hi(v[1]), acc[3]);
                    }
                *reinterpret_cast<u32x2 *>(Z + (uint32_t)px * PZ + (uint32_t)c * 2) =
                    cz ? u32x2{T::pack2(acc[0], acc[1]), T::pack2(acc[2], acc[3])} : u32x2{0u, 0u};
            }

            // 4. the FFN
            u32x4 zf[KS];
#pragma unroll
            for (int ks = 0; ks < KS; ks++)
                zf[ks] = *reinterpret_cast<const u32x4 *>(Z + (uint32_t)jl * PZ + (uint32_t)(32 * ks + 8 * q) * 2);
            float4v acc_o[OTM];
#pragma unroll
            for (int ot = 0; ot < OTM; ot++)
                acc_o[ot] = float4v{0.f, 0.f, 0.f, 0.f};
            auto chunk = [&](int kk) {
                u32x4 w1f[2][KS], w2f[OTM];
                if constexpr (WL) {
                    // the fragments straight from the staged rows (clamped)
#pragma unroll
                    for (int t = 0; t < 2; t++) {
                        const uint8_t *wr =
                            smem + a.off_w1 + (uint32_t)min(32 * kk + 16 * t + jl, R - 1) * w1_stride(C);
#pragma unroll
                        for (int ks = 0; ks < KS; ks++) {
                            const int k = 32 * ks + 8 * q;
                            w1f[t][ks] = *reinterpret_cast<const u32x4 *>(wr + (k < C2 ? k : 0) * 2);
                        }
                    }
                    const int ha = 32 * kk + 4 * q, hb = ha + 16 < R ? ha + 16 : ha;
#pragma unroll
                    for (int ot = 0; ot < OTM; ot++)
                        if (ot < OT) {
                            const uint8_t *wr =
                                smem + a.off_w2 + (uint32_t)min(16 * ot + jl, K - 1) * w2_stride(R);
                            const u32x2 pa = *reinterpret_cast<const u32x2 *>(wr + ha * 2),
                                        pb = *reinterpret_cast<const u32x2 *>(wr + hb * 2);
                            w2f[ot] = u32x4{pa[0], pa[1], pb[0], pb[1]};
                        }
                } else {
                    // the fragments from the row-major pieces; then the next
                    // chunk's pieces are loaded into the same registers
#pragma unroll
                    for (int t = 0; t < 2; t++)
#pragma unroll
                        for (int ks = 0; ks < KS; ks++)
#pragma unroll
                            for (int d = 0; d < 4; d++)
                                w1f[t][ks][d] = perm(pidx, f.w1[t][ks][d]);
#pragma unroll
                    for (int ot = 0; ot < OTM; ot++)
                        if (ot < OT)
#pragma unroll
                            for (int d = 0; d < 4; d++)
                                w2f[ot][d] = perm(pidx, f.w2[ot][d >> 1][d & 1]);
                    load_frag(a, min(kk + 1, NKK - 1), lr, lp, f);
                }
                uint32_t hp[4];
#pragma unroll
                for (int t = 0; t < 2; t++) {
                    const int h0 = 32 * kk + 16 * t;  // the expand tile's first hidden channel
                    float4v u = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int ks = 0; ks < KS; ks++)
                        u = T::mfma(w1f[t][ks], zf[ks], u);
                    // lane (q, jl) holds hidden h0 + 4q + e of pixel jl; the
                    // tile past R (R % 32 == 16) is zero
                    const bool live = h0 < R;  // wave-uniform
                    const int hh = live ? h0 + 4 * q : 0;
                    const float4v sc = *reinterpret_cast<const float4v *>(s1l + hh),
                                  bi = *reinterpret_cast<const float4v *>(b1l + hh);
#pragma unroll
                    for (int e2 = 0; e2 < 2; e2++) {
                        float v[2];
#pragma unroll
                        for (int s = 0; s < 2; s++) {
                            const int e = 2 * e2 + s;
                            v[s] = live ? act_f(fmaf(u[e], sc[e], bi[e]), a.act) : 0.0f;
                        }
                        hp[2 * t + e2] = T::pack2(v[0], v[1]);
                    }
                }
                const u32x4 ub = {hp[0], hp[1], hp[2], hp[3]};
#pragma unroll
                for (int ot = 0; ot < OTM; ot++)
                    if (ot < OT)
                        acc_o[ot] = T::mfma(w2f[ot], ub, acc_o[ot]);
            };
#pragma unroll 1
            for (int kk = 0; kk < NKK; kk++)
                chunk(kk);
            // y = s2 * acc + b2: lane (q, jl) holds channels 16 ot + 4q .. + 3 of pixel j0 + jl
            if (j0 + jl < a.Wo) {
                uint16_t *yp = a.y + (((size_t)un.n * a.Ho + i) * a.Wo + j0 + jl) * K;
#pragma unroll
                for (int ot = 0; ot < OTM; ot++) {
                    const int o = 16 * ot + 4 * q;
                    if (o >= K)
                        continue;
                    float r[4];
#pragma unroll
                    for (int e = 0; e < 4; e++)
                        r[e] = fmaf(acc_o[ot][e], s2l[o + e], b2l[o + e]);
                    *reinterpret_cast<u32x2 *>(yp + o) = u32x2{T::pack2(r[0], r[1]), T::pack2(r[2], r[3])};
                }
            }
            if (next >= a.units)
                break;
            unit = next;
            if (!PREF)
                load_window(a, unit, ln, xv);
        }
    }
};

template <typename T, int C, int OTM, bool WL>
__global__ __launch_bounds__(256) void cfs2_kernel(Args a) {
    extern __shared__ __attribute__((aligned(256))) uint8_t smem[];
    Kern<T, C, OTM, WL>::run(a, smem);
}

inline uint32_t region_for(int C) {
    switch (C) {
    case 16: return Kern<F16, 16, 4, false>::REGION;
    case 24: return Kern<F16, 24, 4, false>::REGION;
    case 32: return Kern<F16, 32, 4, false>::REGION;
    case 48: return Kern<F16, 48, 4, false>::REGION;
    case 64: return Kern<F16, 64, 4, false>::REGION;
    default: return 0;
    }
}

// waves per workgroup (1 .. 4): the count that lets a compute unit's LDS
// hold the most waves (every workgroup stages its own taps and vectors, and
// the weights when wl); 0 when not even one wave fits.  *per_cu receives
// that many waves.
inline int waves_for(int C, int R, int K, bool wl, int *per_cu = nullptr) {
    const uint32_t r = region_for(C), lds = 160u * 1024u;
    const uint32_t st = staged_bytes(C, R, K) + (wl ? weights_bytes(C, R, K) : 0u);
    int best = 0, best_waves = 0;
    for (int nw = 1; r && nw <= 4; nw++) {
        const uint32_t wg = st + (uint32_t)nw * r;
        const int waves = wg <= lds ? nw * (int)(lds / wg) : 0;
        if (waves >= best_waves && waves > 0) {
            best = nw;
            best_waves = waves;
        }
    }
    if (per_cu)
        *per_cu = best_waves;
    return best;
}

// the weights go to LDS when that still leaves two waves per SIMD, or as
// many waves as without them (measured: at 128 x 128 x 16, 8 waves with the
// weights in LDS beat 10 without; at 64 x 64 x 32, 4 lose to 6)
inline bool weights_in_lds(int C, int R, int K) {
    int wl = 0, wg = 0;
    waves_for(C, R, K, true, &wl);
    waves_for(C, R, K, false, &wg);
    return wl >= 1 && (wl >= 8 || wl >= wg);
}

template <typename T, int C, int OTM, bool WL>
hipError_t launch_t(const Args &a, size_t lds, int grid, hipStream_t st) {
    auto kf = cfs2_kernel<T, C, OTM, WL>;
    hipError_t e = allow_full_lds((const void *)kf);
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(kf, dim3(grid), dim3(64 * a.nw), lds, st, a);
    return hipGetLastError();
}

template <typename T, int C, bool WL>
hipError_t launch_w(const Args &a, size_t lds, int grid, hipStream_t st) {
    if (a.K <= 32)
        return launch_t<T, C, 2, WL>(a, lds, grid, st);
    return a.K <= 64 ? launch_t<T, C, 4, WL>(a, lds, grid, st) : launch_t<T, C, 8, WL>(a, lds, grid, st);
}

template <typename T, int C>
hipError_t launch_k(const Args &a, bool wl, size_t lds, int grid, hipStream_t st) {
    return wl ? launch_w<T, C, true>(a, lds, grid, st) : launch_w<T, C, false>(a, lds, grid, st);
}

template <typename T>
hipError_t launch_c(const Args &a, int C, bool wl, size_t lds, int grid, hipStream_t st) {
    switch (C) {
    case 16: return launch_k<T, 16>(a, wl, lds, grid, st);
    case 24: return launch_k<T, 24>(a, wl, lds, grid, st);
    case 32: return launch_k<T, 32>(a, wl, lds, grid, st);
    case 48: return launch_k<T, 48>(a, wl, lds, grid, st);
    case 64: return launch_k<T, 64>(a, wl, lds, grid, st);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace cfs2

bool convfirst_s2_supported(int H, int W, int C, int R, int K) {
    return H >= 2 && W >= 2 && R >= 16 && R % 16 == 0 && R <= cfs2::RMAX && K >= 8 && K % 8 == 0 &&
           K <= cfs2::KMAX && cfs2::waves_for(C, R, K, false) >= 1;
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
    const bool wl = cfs2::weights_in_lds(C, R, K);
    a.nw = cfs2::waves_for(C, R, K, wl);
    a.off_w1 = cfs2::staged_bytes(C, R, K);
    a.off_w2 = a.off_w1 + (uint32_t)R * cfs2::w1_stride(C);
    a.off_region = a.off_w1 + (wl ? cfs2::weights_bytes(C, R, K) : 0u);
    const size_t lds = a.off_region + (size_t)a.nw * cfs2::region_for(C);
    // persistent workgroups: as many as the LDS lets every compute unit hold
    const int per_cu = (int)((160u * 1024u) / lds);
    const int64_t need = (a.units + a.nw - 1) / a.nw;
    const int64_t cap = (int64_t)(per_cu > 0 ? per_cu : 1) * device_cu_count();
    const int grid = (int)(need < cap ? need : cap);
    return bf16 ? cfs2::launch_c<BF16>(a, C, wl, lds, grid, st) : cfs2::launch_c<F16>(a, C, wl, lds, grid, st);
}

}  // namespace cf
