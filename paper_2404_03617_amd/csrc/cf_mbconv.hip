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
//  1. expand: the group's 64 rows of W1 (in LDS for the whole launch)
//     against every pixel of the image (v_mfma_f32_16x16x32, x read straight
//     from global memory as B fragments in batches of four K steps), SiLU in
//     fp32, rounded into an LDS buffer with a zero border;
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
//  6. the projection: the image's output is cut into units of 16 pixels and
//     a range of 16-channel tiles, dealt round-robin to the image's work
//     items; a unit's 16 pixels of V, times the gates, are read once into LDS
//     and every tile of the unit is a product over all E*C hidden channels of
//     W2 rows (batches of eight K steps, the next batch in flight) and the
//     staged V; then s3, b3 and the residual, and y is written once.  The
//     conv taps stay in registers and the scale/bias vectors in LDS for the
//     whole launch.
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
// read.  Each slot has a line in the workspace header (arrivals, give-up,
// exits) that its last work item zeroes on the way out, so a call is one
// launch and the header, zeroed once before first use, stays zero between
// calls whatever shapes share the workspace.  The wait is bounded; one that
// gives up sets a flag in the workspace, the slot's later waits of the call
// are skipped, and the kernel always ends.
//
// Images up to 16 x 16 (the late-stage shapes the paper targets); C a
// multiple of 16; E*C a multiple of 64 and at most 4096; 1 <= R <= 256; the
// LDS layout within 160 KB (it grows with C and E*C: C up to 768 at E = 2,
// 512 at E = 4, 256 at E = 8).
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
constexpr int SLOTMAX = 2048;     // images in flight the workspace header has lines for

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
    int *flag;                     // set to 1 when a barrier wait gives up (never cleared here)
    int *line;                     // [SLOTMAX][32]: per slot arrivals, give-up, exits (zero between calls)
    float *sq;                     // [N][G][R] squeeze shares
    uint16_t *vx;                  // [2][slots][Po][EC] exchanged conv output (stride 2: after BlurPool)
    int N, H, W, C, EC, R, G;
    int K, Ho, Wo;                 // output channels and size (stride 1: C, H, W)
    uint32_t off_vb;               // stride 2: LDS copy of the group's conv output [H*W][PB]
    int slots;
    int xcd_map;                   // 1: the workgroups of a slot share an XCD
    uint32_t off_gate, off_z, off_cs, off_vec, off_w1;  // LDS layout (U at 0)
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

// Barrier of a slot's work items at the end of their `target` / G-th image:
// every thread's device-scope stores so far are complete when the workgroup
// adds its arrival to the slot's count (it grows by G per image); returns once
// the count reaches `target`.  The wait is bounded: a work item that gives up
// marks the slot's line (the slot's later waits in this call are then
// skipped) and sets the workspace flag, which stays set for the caller.
__device__ __forceinline__ void slot_barrier(const Args &a, int *line, int target) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (threadIdx.x == 0) {
        __hip_atomic_fetch_add(line, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        int spins = 0;
        while (__hip_atomic_load(line, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
            const bool over = ++spins > SPIN_LIMIT;
            if (over || ((spins & 63) == 1 && __hip_atomic_load(line + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))) {
                if (over) {
                    __hip_atomic_store(line + 1, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    __hip_atomic_store(a.flag, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                }
                break;
            }
            __builtin_amdgcn_s_sleep(1);
        }
    }
    __syncthreads();
}

// After its last image a work item adds its exit to the slot's line; the last
// of the slot's G exits (every wait of the slot is over) zeroes the line, so
// each call leaves the header as it found it.
__device__ __forceinline__ void slot_exit(int *line, int G) {
    if (threadIdx.x == 0 && __hip_atomic_fetch_add(line + 2, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == G - 1) {
        __hip_atomic_store(line, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(line + 1, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(line + 2, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

template <typename T, int NWV, int NPW, bool S2 = false>
struct MB {
    static constexpr int NT = NWV * 64;
    static constexpr int NGG = 8 / NWV;  // 8-channel conv groups per wave
    static constexpr int KE = NPW == 4 ? 2 : 4;  // expand K steps per load batch
    static constexpr int KB = NPW == 2 ? 8 : 4;  // output K steps per load batch (two batches in flight)

    static __device__ void run(const Args &a, uint8_t *smem) {
        const int tid = threadIdx.x, lane = tid & 63;
        const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
        const int q = lane >> 4, jl = lane & 15;
        // Fragments read straight from global memory (x in the expand, W2 in
        // the projection) are loaded with four adjacent lanes on 64
        // contiguous bytes of one row (lane l: row l / 4, piece l % 4) -- the
        // memory unit merges only adjacent lanes, and in fragment order every
        // lane would start a row of its own -- and each dword then moves to
        // its fragment lane (q, jl), which takes row jl, piece q from lane
        // 4 jl + q
        const int lr = lane >> 2, lp = lane & 3;
        const int perm = (4 * jl + q) * 4;  // ds_bpermute source address
        auto permute = [&](const u32x4 &v) {
            u32x4 o;
#pragma unroll
            for (int d = 0; d < 4; d++)
                o[d] = (uint32_t)__builtin_amdgcn_ds_bpermute(perm, (int)v[d]);
            return o;
        };
        const int M = gridDim.x;
        int lin = blockIdx.x;
        if (a.xcd_map)  // workgroup i runs on XCD i % 8
            lin = (int)(blockIdx.x % 8) * (M / 8) + (int)(blockIdx.x / 8);
        const int g = lin % a.G, slot = lin / a.G;
        const int C = a.C, EC = a.EC, R = a.R, G = a.G;
        const int P = a.H * a.W;
        const int Po = S2 ? a.Ho * a.Wo : P;  // output pixels
        const int KO = S2 ? a.K : C;           // output channels
        const int RP = (a.H + 1) / 2;
        const int h0 = g * GH;  // first hidden channel of the group
        uint8_t *U = smem;
        float *gate = reinterpret_cast<float *>(smem + a.off_gate);  // [EC]
        float *zl = reinterpret_cast<float *>(smem + a.off_z);       // [R]
        float *csum = reinterpret_cast<float *>(smem + a.off_cs);    // [64]
        float *vec = reinterpret_cast<float *>(smem + a.off_vec);    // s1, b1, s2, b2 [64] each; s3, b3 [C]
        float *s1l = vec, *b1l = vec + 64, *s2l = vec + 128, *b2l = vec + 192, *s3l = vec + 256, *b3l = s3l + KO;
        int *line = a.line + 32 * (size_t)slot;

        // once per workgroup: the scale/bias vectors the group uses
        for (int i = tid; i < 64; i += NT) {
            s1l[i] = a.s1 ? a.s1[h0 + i] : 1.0f;
            b1l[i] = a.b1 ? a.b1[h0 + i] : 0.0f;
            s2l[i] = a.s2 ? a.s2[h0 + i] : 1.0f;
            b2l[i] = a.b2 ? a.b2[h0 + i] : 0.0f;
        }
        for (int i = tid; i < KO; i += NT) {
            s3l[i] = a.s3 ? a.s3[i] : 1.0f;
            b3l[i] = a.b3 ? a.b3[i] : 0.0f;
        }
        // the group's 64 rows of W1 (pitch 2C + 16 bytes: an odd multiple of
        // 16, conflict-free fragment reads)
        const uint32_t w1p = 2 * C + 16;
        uint8_t *w1l = smem + a.off_w1;
        for (int i = tid; i < 64 * (C / 8); i += NT) {
            const int row = i / (C / 8), c8 = i - row * (C / 8);
            *reinterpret_cast<u32x4 *>(w1l + (uint32_t)row * w1p + (uint32_t)c8 * 16) =
                ld16(a.w1 + (size_t)(h0 + row) * C + 8 * c8);
        }
        // the conv taps of this wave's 8-channel groups stay in registers
        const int cs = jl >> 3, co = jl & 7;
        const int ti = q - cs;  // the tap row this lane's K slice meets
        const bool tap_ok = ti >= 0 && ti <= 2;
        u32x4 cav[NGG][3];
#pragma unroll
        for (int j = 0; j < NGG; j++)
#pragma unroll
            for (int dj = 0; dj < 3; dj++)
                cav[j][dj] = tap_ok ? ld16(a.gw + ((size_t)(ti * 3 + dj) * EC + h0 + 8 * (wv + NWV * j) + co) * 8)
                                    : u32x4{0u, 0u, 0u, 0u};
        __syncthreads();

        int it = 0;
        for (int n = slot; n < a.N; n += a.slots, it++) {
            const uint16_t *xn = a.x + (size_t)n * P * C;
            uint16_t *vx = a.vx + ((size_t)(it & 1) * a.slots + slot) * Po * EC;

            // the U border (row 0, rows past H, column 0, columns past W) is
            // zero; the output staging of the previous image overwrote it
            {
                const int urows = 2 * RP + 2;
                for (int i = tid; i < urows * UC * (PB / 16); i += NT) {
                    const int cell = i / (PB / 16), row = cell / UC, col = cell - row * UC;
                    if (row == 0 || row > a.H || col == 0 || col > a.W)
                        *reinterpret_cast<u32x4 *>(U + (uint32_t)i * 16) = u32x4{0u, 0u, 0u, 0u};
                }
            }

            // ---- 1. expand + SiLU into U; wave wv takes the 16-pixel tiles wv + NWV i
            {
                float4v acc[4][NPW];
#pragma unroll
                for (int mt = 0; mt < 4; mt++)
#pragma unroll
                    for (int i = 0; i < NPW; i++)
                        acc[mt][i] = float4v{0.f, 0.f, 0.f, 0.f};
                const int ks = (C + 31) / 32;
                for (int k0 = 0; k0 < ks; k0 += KE) {
                    u32x4 bv[KE][NPW];
#pragma unroll
                    for (int j = 0; j < KE; j++) {
                        const int k = 32 * (k0 + j) + 8 * lp;
                        const bool kin = k < C;  // past ks, or the half-padded last step of C % 32 == 16
#pragma unroll
                        for (int i = 0; i < NPW; i++) {
                            const int p = 16 * (wv + NWV * i) + lr;
                            bv[j][i] = kin && p < P ? ld16(xn + (size_t)p * C + k) : u32x4{0u, 0u, 0u, 0u};
                        }
                    }
#pragma unroll
                    for (int j = 0; j < KE; j++)
#pragma unroll
                        for (int i = 0; i < NPW; i++)
                            bv[j][i] = permute(bv[j][i]);
#pragma unroll
                    for (int j = 0; j < KE; j++) {
                        if (k0 + j >= ks)  // wave-uniform
                            break;
                        const int k = 32 * (k0 + j) + 8 * q;
#pragma unroll
                        for (int mt = 0; mt < 4; mt++) {
                            // A rows of W1; a K slice past C multiplies zero x
                            const u32x4 av = k < C ? *reinterpret_cast<const u32x4 *>(
                                                         w1l + (uint32_t)(16 * mt + jl) * w1p + (uint32_t)k * 2)
                                                   : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
                            for (int i = 0; i < NPW; i++)
                                acc[mt][i] = T::mfma(av, bv[j][i], acc[mt][i]);
                        }
                    }
                }
#pragma unroll
                for (int mt = 0; mt < 4; mt++) {
                    const int hl = 16 * mt + 4 * q;  // local hidden channels hl .. hl+3 of this lane
                    const float4v sc = *reinterpret_cast<const float4v *>(s1l + hl);
                    const float4v bi = *reinterpret_cast<const float4v *>(b1l + hl);
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
#pragma unroll
            for (int j = 0; j < NGG; j++) {
                const int gg = wv + NWV * j;
                const int hl = 8 * gg + 4 * (q & 1);  // output channels of this lane's D rows
                const float4v sc = *reinterpret_cast<const float4v *>(s2l + hl);
                const float4v bi = *reinterpret_cast<const float4v *>(b2l + hl);
                float sum[4] = {0.f, 0.f, 0.f, 0.f};
                for (int rp = 0; rp < RP; rp++) {
                    float4v acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int dj = 0; dj < 3; dj++) {
                        const u32x4 bv = *reinterpret_cast<const u32x4 *>(
                            U + (uint32_t)((2 * rp + q) * UC + jl + dj) * PB + (uint32_t)gg * 16);
                        acc = T::mfma(cav[j][dj], bv, acc);
                    }
                    const int r = 2 * rp + (q >> 1), c = jl;
                    if (r < a.H && c < a.W) {
                        float u[4];
#pragma unroll
                        for (int e = 0; e < 4; e++) {
                            u[e] = silu_f32(fmaf(acc[e], sc[e], bi[e]));
                            sum[e] += u[e];
                        }
                        const u32x2 pk = {T::pack2(u[0], u[1]), T::pack2(u[2], u[3])};
                        if constexpr (S2)  // the group's copy in LDS, for the BlurPool below
                            *reinterpret_cast<u32x2 *>(smem + a.off_vb + (uint32_t)(r * a.W + c) * PB +
                                                       (uint32_t)hl * 2) = pk;
                        else
                            st8_dev(vx + (size_t)(r * a.W + c) * EC + h0 + hl, pk);
                    }
                }
                if constexpr (S2)
                    continue;  // the channel sums are those of the down-sampled map (below)
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
            __syncthreads();

            if constexpr (S2) {
                // ---- 2b. BlurPool of the group's 64 channels (Triangle-3 taps
                //      [1, 2, 1] / 4 in each direction, one pixel of reflect
                //      padding, stride 2) from the LDS copy of V, rounded V'
                //      to the exchange buffer; the channel sums of V' (fp32,
                //      before rounding) in a fixed order: per thread over its
                //      pixels, then over the threads through the free U area
                float *part = reinterpret_cast<float *>(U);  // [NT / 16][64]
                constexpr int NPG = NT / 16;
                const int c4 = tid & 15, pg = tid >> 4;  // channels 4 c4 .. 4 c4 + 3
                const uint8_t *vb = smem + a.off_vb + (uint32_t)c4 * 8;
                float s4[4] = {0.f, 0.f, 0.f, 0.f};
                for (int pp = pg; pp < Po; pp += NPG) {
                    const int i = pp / a.Wo, j = pp - i * a.Wo;
                    float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int ta = 0; ta < 3; ta++) {
                        int r = 2 * i + ta - 1;
                        r = r < 0 ? -r : (r >= a.H ? 2 * (a.H - 1) - r : r);
#pragma unroll
                        for (int tb = 0; tb < 3; tb++) {
                            int c = 2 * j + tb - 1;
                            c = c < 0 ? -c : (c >= a.W ? 2 * (a.W - 1) - c : c);
                            const float wt = (ta == 1 ? 0.5f : 0.25f) * (tb == 1 ? 0.5f : 0.25f);
                            const u32x2 v = *reinterpret_cast<const u32x2 *>(vb + (uint32_t)(r * a.W + c) * PB);
                            acc[0] = fmaf(wt, T::lo(v[0]), acc[0]);
                            acc[1] = fmaf(wt, T::hi(v[0]), acc[1]);
                            acc[2] = fmaf(wt, T::lo(v[1]), acc[2]);
                            acc[3] = fmaf(wt, T::hi(v[1]), acc[3]);
                        }
                    }
#pragma unroll
                    for (int e = 0; e < 4; e++)
                        s4[e] += acc[e];
                    st8_dev(vx + (size_t)pp * EC + h0 + 4 * c4,
                            u32x2{T::pack2(acc[0], acc[1]), T::pack2(acc[2], acc[3])});
                }
#pragma unroll
                for (int e = 0; e < 4; e++)
                    part[pg * 64 + 4 * c4 + e] = s4[e];
                __syncthreads();
                if (tid < 64) {
                    float sm = 0.0f;
                    for (int g2 = 0; g2 < NPG; g2++)
                        sm += part[g2 * 64 + tid];
                    csum[tid] = sm;
                }
                __syncthreads();
            }

            // ---- 3. the group's share of the squeeze: Wr[:, group] . mean(V)
            if (tid < R) {
                const float inv = 1.0f / (float)Po;
                float s = 0.0f;
                const uint16_t *wrow = a.wr + (size_t)tid * EC + h0;
                Pack8 w[GH / 8];
#pragma unroll
                for (int c = 0; c < GH / 8; c++)
                    w[c].u = ld16(wrow + 8 * c);
#pragma unroll
                for (int c = 0; c < GH / 8; c++)
#pragma unroll
                    for (int e = 0; e < 4; e++)
                        s += T::lo(w[c].w[e]) * csum[8 * c + 2 * e] + T::hi(w[c].w[e]) * csum[8 * c + 2 * e + 1];
                __hip_atomic_store(a.sq + ((size_t)n * G + g) * R + tid, s * inv, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
            }

            // ---- 4. every work item of image n has written its V and its share
            slot_barrier(a, line, G * (it + 1));

            // ---- 5. squeeze (shares in group order), excitation, gates of all channels
            for (int r = tid; r < R; r += NT) {
                const float *sp = a.sq + (size_t)n * G * R + r;
                float s = a.br ? a.br[r] : 0.0f;
                int gg = 0;
                for (; gg + 8 <= G; gg += 8) {
                    float v[8];
#pragma unroll
                    for (int u = 0; u < 8; u++)
                        v[u] = __hip_atomic_load(sp + (size_t)(gg + u) * R, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
                    for (int u = 0; u < 8; u++)
                        s += v[u];
                }
                for (; gg < G; gg++)
                    s += __hip_atomic_load(sp + (size_t)gg * R, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                zl[r] = s > 0.0f ? s : 0.0f;
            }
            __syncthreads();
            for (int c = tid; c < EC; c += NT) {
                const uint16_t *wrow = a.we + (size_t)c * R;
                float s = a.be ? a.be[c] : 0.0f;
                int r = 0;
                if ((R & 7) == 0) {
                    for (; r + 64 <= R; r += 64) {  // eight 16-byte loads in flight
                        Pack8 w[8];
#pragma unroll
                        for (int u = 0; u < 8; u++)
                            w[u].u = ld16(wrow + r + 8 * u);
#pragma unroll
                        for (int u = 0; u < 8; u++)
#pragma unroll
                            for (int e = 0; e < 4; e++)
                                s += T::lo(w[u].w[e]) * zl[r + 8 * u + 2 * e] +
                                     T::hi(w[u].w[e]) * zl[r + 8 * u + 2 * e + 1];
                    }
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

            // ---- 6. output.  The image's pixel tiles x output-channel tiles are
            //      cut into units of one pixel tile and a range of channel
            //      tiles, dealt round-robin to the image's work items (more
            //      channel ranges per pixel tile when the work items outnumber
            //      the pixel tiles, so a work item then has one unit; otherwise
            //      every unit spans all channel tiles).  The work item's units
            //      of V, times the gates, are staged in LDS over the dead U
            //      buffer; each channel tile is a product over all EC hidden
            //      channels of W2 rows (loaded in batches of KB steps, the next
            //      batch in flight, each fragment serving two units) and the
            //      staged V; then s3, b3 and the residual, and y is written once.
            {
                const int PT = (Po + 15) / 16, OT = KO / 16;
                const int NOG = G > PT ? G / PT : 1;
                const int per = (OT + NOG - 1) / NOG;  // channel tiles per unit
                const int units = PT * NOG;
                const int nu = g < units ? (units - g + G - 1) / G : 0;  // units g + G u of this work item
                const int ot0 = NOG > 1 ? (g / PT) * per : 0, ot1 = min(OT, ot0 + per);
                const int kst = EC / 32;
                const int nbat = (kst + KB - 1) / KB;
                const uint32_t pitch = 2 * EC + 16;  // staged bytes per pixel: an odd multiple of 16
                const int c4n = EC / 4;
                // stage the gated V of every unit (zero past P)
                for (int idx = tid; idx < nu * 16 * c4n; idx += NT) {
                    const int row = idx / c4n, c4 = idx - row * c4n;  // row = 16 u + pixel
                    const int p = 16 * ((g + G * (row >> 4)) % PT) + (row & 15);
                    u32x2 v = {0u, 0u};
                    if (p < Po) {
                        const u32x2 raw = ld8_dev(vx + (size_t)p * EC + 4 * c4);
                        const float4v gv = *reinterpret_cast<const float4v *>(gate + 4 * c4);
                        v[0] = T::pack2(T::lo(raw[0]) * gv[0], T::hi(raw[0]) * gv[1]);
                        v[1] = T::pack2(T::lo(raw[1]) * gv[2], T::hi(raw[1]) * gv[3]);
                    }
                    *reinterpret_cast<u32x2 *>(U + (uint32_t)row * pitch + (uint32_t)c4 * 8) = v;
                }
                __syncthreads();
                for (int u0 = 0; u0 < nu; u0 += 2) {
                    const bool two = u0 + 1 < nu;  // wave-uniform
                    const int p0 = 16 * ((g + G * u0) % PT) + jl;
                    const int p1 = 16 * ((g + G * (u0 + 1)) % PT) + jl;
                    const uint8_t *vl0 = U + (uint32_t)(16 * u0 + jl) * pitch + (uint32_t)q * 16;
                    const uint8_t *vl1 = vl0 + 16 * pitch;
                    for (int ot = ot0 + wv; ot < ot1; ot += NWV) {
                        const uint16_t *wrow = a.w2 + (size_t)(16 * ot + lr) * EC + 8 * lp;
                        const int o = 16 * ot + 4 * q;
                        u32x2 xv0 = {0u, 0u}, xv1 = {0u, 0u};  // the residual (stride 1 only)
                        if (!S2 && p0 < P)
                            xv0 = *reinterpret_cast<const u32x2 *>(a.x + ((size_t)n * P + p0) * C + o);
                        if (!S2 && two && p1 < P)
                            xv1 = *reinterpret_cast<const u32x2 *>(a.x + ((size_t)n * P + p1) * C + o);
                        float4v acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
                        auto loadb = [&](int b, u32x4 *w) {
#pragma unroll
                            for (int j = 0; j < KB; j++) {
                                const int kk = KB * b + j;
                                if (kk < kst)
                                    w[j] = ld16(wrow + 32 * kk);
                            }
                        };
                        auto mmab = [&](int b, const u32x4 *w) {
#pragma unroll
                            for (int j = 0; j < KB; j++) {
                                const int kk = KB * b + j;
                                if (kk >= kst)
                                    break;
                                const u32x4 wf = permute(w[j]);
                                acc0 = T::mfma(wf, *reinterpret_cast<const u32x4 *>(vl0 + (uint32_t)kk * 64), acc0);
                                if (two)
                                    acc1 = T::mfma(wf, *reinterpret_cast<const u32x4 *>(vl1 + (uint32_t)kk * 64),
                                                   acc1);
                            }
                        };
                        u32x4 wA[KB], wB[KB];
                        loadb(0, wA);
                        for (int b = 0; b < nbat; b += 2) {
                            if (b + 1 < nbat)
                                loadb(b + 1, wB);
                            mmab(b, wA);
                            if (b + 1 < nbat) {
                                if (b + 2 < nbat)
                                    loadb(b + 2, wA);
                                mmab(b + 1, wB);
                            }
                        }
                        const float4v sc = *reinterpret_cast<const float4v *>(s3l + o);
                        const float4v bi = *reinterpret_cast<const float4v *>(b3l + o);
                        auto store = [&](int p, const u32x2 &xv, const float4v &acc) {
                            u32x2 out;
                            out[0] = T::pack2(T::lo(xv[0]) + fmaf(acc[0], sc[0], bi[0]),
                                              T::hi(xv[0]) + fmaf(acc[1], sc[1], bi[1]));
                            out[1] = T::pack2(T::lo(xv[1]) + fmaf(acc[2], sc[2], bi[2]),
                                              T::hi(xv[1]) + fmaf(acc[3], sc[3], bi[3]));
                            *reinterpret_cast<u32x2 *>(a.y + ((size_t)n * Po + p) * KO + o) = out;
                        };
                        if (p0 < Po)
                            store(p0, xv0, acc0);
                        if (two && p1 < Po)
                            store(p1, xv1, acc1);
                    }
                }
                __syncthreads();  // the staging area is U again for the next image
            }
            // the next image rewrites U (its border first, then the interior)
            // after the __syncthreads that ends the last unit above
        }
        slot_exit(line, G);
    }
};

// registers for two waves per SIMD: one 8-wave or two 4-wave workgroups per
// CU (the LDS layout of three or more would not fit with W1 resident)
template <typename T, int NWV, int NPW, bool S2 = false>
__global__ __launch_bounds__(NWV * 64) __attribute__((amdgpu_waves_per_eu(2))) void mbconv_kernel(Args a) {
    extern __shared__ __attribute__((aligned(256))) uint8_t smem[];
    MB<T, NWV, NPW, S2>::run(a, smem);
}

struct Layout {
    uint32_t off_gate, off_z, off_cs, off_vec, off_w1, off_vb, lds;
    int nwv;
};

// LDS layout for an H x W image.  U holds the border row above the image,
// its H rows, and zero rows below up to an even count of row pairs plus one
// (the conv reads halo rows 2rp .. 2rp+3 for every row pair rp); the output
// phase stages the work item's units of gated V over the same bytes.  Then
// the gates of all EC channels, the squeeze vector, the group's channel sums,
// the fp32 scale/bias vectors (the group's s1, b1, s2, b2; all of s3, b3) and
// the group's rows of W1; for stride 2 (K > 0 output channels) last the
// group's copy of the full-resolution conv output.
Layout layout(int H, int W, int C, int EC, int R, int K = 0) {
    Layout l;
    const int P = H * W, Po = K > 0 ? ((H + 1) / 2) * ((W + 1) / 2) : P, KO = K > 0 ? K : C;
    const int G = EC / GH, PT = (Po + 15) / 16;
    const uint32_t urows = (uint32_t)(2 * ((H + 1) / 2) + 2);
    const uint32_t nu = G > PT ? 1 : (uint32_t)((PT + G - 1) / G);  // output units of a work item
    const uint32_t ubytes = urows * UC * PB, stage = nu * 16 * (2 * (uint32_t)EC + 16);
    l.off_gate = ubytes > stage ? ubytes : stage;
    l.off_z = l.off_gate + (uint32_t)EC * 4;
    l.off_cs = l.off_z + (((uint32_t)R * 4 + 15) & ~15u);
    l.off_vec = l.off_cs + GH * 4;
    l.off_w1 = l.off_vec + (4 * GH + 2 * (uint32_t)KO) * 4;
    l.off_vb = l.off_w1 + 64 * (2 * (uint32_t)C + 16);
    l.lds = l.off_vb + (K > 0 ? (uint32_t)P * PB : 0u);
    // 4-wave workgroups, two or more per CU; 8-wave ones for 16 x 16 images
    // whose layout leaves room for only one workgroup
    l.nwv = P > 128 && l.lds > 80 * 1024 ? 8 : 4;
    return l;
}

size_t head_bytes() { return 256 + (size_t)SLOTMAX * 128; }
size_t sq_bytes(int N, int G, int R) { return ((size_t)N * G * R * 4 + 255) & ~(size_t)255; }

}  // namespace mbc

bool mbconv_supported(int H, int W, int C, int E, int R, int K) {
    return H >= (K > 0 ? 2 : 1) && W >= (K > 0 ? 2 : 1) && H <= mbc::HMAX && W <= mbc::WMAX && C >= 16 &&
           C % 16 == 0 && E >= 1 && (E * C) % mbc::GH == 0 && E * C <= mbc::ECMAX && R >= 1 && R <= mbc::RMAX &&
           K >= 0 && K % 16 == 0 && K <= mbc::ECMAX && mbc::layout(H, W, C, E * C, R, K).lds <= 160 * 1024;
}

namespace {

// The kernel instance for the shape and its launch size.
template <bool S2>
const void *kernel_s(int nwv, int P, int bf16) {
    if (nwv == 8)
        return bf16 ? (const void *)mbc::mbconv_kernel<BF16, 8, 2, S2> : (const void *)mbc::mbconv_kernel<F16, 8, 2, S2>;
    if (P > 128)
        return bf16 ? (const void *)mbc::mbconv_kernel<BF16, 4, 4, S2> : (const void *)mbc::mbconv_kernel<F16, 4, 4, S2>;
    if (P > 64)
        return bf16 ? (const void *)mbc::mbconv_kernel<BF16, 4, 2, S2> : (const void *)mbc::mbconv_kernel<F16, 4, 2, S2>;
    return bf16 ? (const void *)mbc::mbconv_kernel<BF16, 4, 1, S2> : (const void *)mbc::mbconv_kernel<F16, 4, 1, S2>;
}

const void *mbconv_kernel_for(int H, int W, int C, int EC, int R, int K, int bf16, mbc::Layout *l, int *nt) {
    *l = mbc::layout(H, W, C, EC, R, K);
    *nt = l->nwv * 64;
    return K > 0 ? kernel_s<true>(l->nwv, H * W, bf16) : kernel_s<false>(l->nwv, H * W, bf16);
}

}  // namespace

hipError_t mbconv_resident_slots(int H, int W, int C, int E, int R, int K, int bf16, int *slots) {
    mbc::Layout l;
    int nt = 0;
    const void *kf = mbconv_kernel_for(H, W, C, E * C, R, K, bf16, &l, &nt);
    hipError_t e = allow_full_lds(kf);
    if (e != hipSuccess)
        return e;
    int per_cu = 0;
    if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kf, nt, l.lds)) != hipSuccess)
        return e;
    *slots = per_cu * device_cu_count() / (E * C / mbc::GH);
    return hipSuccess;
}

// pixels of the exchanged map: the block's output size
static size_t mbconv_out_pixels(int H, int W, int K) {
    return K > 0 ? (size_t)((H + 1) / 2) * ((W + 1) / 2) : (size_t)H * W;
}

size_t mbconv_workspace_bytes(int N, int H, int W, int C, int E, int R, int K, int slots) {
    const int G = E * C / mbc::GH;
    return mbc::head_bytes() + mbc::sq_bytes(N, G, R) + 2 * (size_t)slots * mbconv_out_pixels(H, W, K) * E * C * 2;
}

hipError_t launch_mbconv(const void *x, void *y, const MBConvW &w, int N, int H, int W, int C, int E, int R, int K,
                         int bf16, void *ws, size_t ws_bytes, bool coop, hipStream_t st) {
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
    a.K = K > 0 ? K : C;
    a.Ho = K > 0 ? (H + 1) / 2 : H;
    a.Wo = K > 0 ? (W + 1) / 2 : W;
    mbc::Layout l;
    int nt = 0;
    const void *kf = mbconv_kernel_for(H, W, C, a.EC, R, K, bf16, &l, &nt);
    a.off_gate = l.off_gate;
    a.off_z = l.off_z;
    a.off_cs = l.off_cs;
    a.off_vec = l.off_vec;
    a.off_w1 = l.off_w1;
    a.off_vb = l.off_vb;
    const size_t fixed = mbc::head_bytes() + mbc::sq_bytes(N, a.G, R);
    const size_t per_slot = 2 * mbconv_out_pixels(H, W, K) * a.EC * 2;
    if (ws_bytes < fixed + per_slot)
        return hipErrorInvalidValue;
    char *base = (char *)ws;
    a.flag = (int *)base;
    a.line = (int *)(base + 256);
    a.sq = (float *)(base + mbc::head_bytes());
    // every work item of an image must be resident with the others (the
    // barrier waits for them): the grid holds at most what fits on the device
    // and is launched cooperatively, which the runtime refuses rather than
    // run partly -- or, for a caller that owns the device, as an ordinary
    // launch, which then starts every workgroup at once
    int slots = 0;
    hipError_t e = mbconv_resident_slots(H, W, C, E, R, K, bf16, &slots);
    if (e != hipSuccess)
        return e;
    if (slots < 1)
        return hipErrorInvalidConfiguration;  // the groups of one image do not fit at once
    if (slots > N)
        slots = N;
    if (slots > mbc::SLOTMAX)
        slots = mbc::SLOTMAX;
    if ((size_t)slots * per_slot > ws_bytes - fixed)
        slots = (int)((ws_bytes - fixed) / per_slot);
    // as few images in flight as the same number of passes over the batch needs
    const int passes = (N + slots - 1) / slots;
    slots = (N + passes - 1) / passes;
    a.slots = slots;
    a.vx = (uint16_t *)(base + fixed);
    const int grid = slots * a.G;
    // a slot's workgroups on one XCD when the grid allows it
    a.xcd_map = grid % 8 == 0 && (grid / 8) % a.G == 0 ? 1 : 0;
    void *args[] = {&a};
    return coop ? hipLaunchCooperativeKernel(kf, dim3(grid), dim3(nt), args, l.lds, st)
                : hipLaunchKernel(kf, dim3(grid), dim3(nt), args, l.lds, st);
}

}  // namespace cf
