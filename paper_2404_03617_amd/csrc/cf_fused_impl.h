// cf_fused_impl.h -- template of the fused ConvFirst block kernel for gfx950;
// instantiated per (C, dtype) in cf_fused_c*.hip so the units compile in
// parallel.
//
// One workgroup (NWAVE waves) owns a tile of M consecutive pixels of the
// flattened N*H*W index and evaluates the whole residual block for it
// (block fusion, Sec. 5.3.1 of Lavin, arXiv:2404.03617):
//   1. the input rows the tile touches plus k/2 halo rows are copied into LDS
//      by asynchronous 16-byte global->LDS loads, in slabs of 64 channels;
//      the copy of the next tile overlaps the FFN of the current one;
//   2. each lane runs the k x k depth-wise conv for its pixels on the VALU
//      (packed fp16 FMA for fp16 I/O, fp32 for bf16) and keeps the result in
//      registers as MFMA B fragments;
//   3. the output accumulators (fp32, registers) start at x + b2, read from
//      the halo tile: the residual shortcut costs no extra HBM read;
//   4. a loop over chunks of 32 hidden channels (eq. e:ffn-eff) computes
//      H^T = W1_chunk D^T on v_mfma_f32_32x32x16 with b1 in the C operand,
//      applies phi, and feeds the converted result straight from the
//      accumulators into the project MFMA  Out^T += W2_chunk H^T: the hidden
//      tile never reaches LDS or HBM;
//   5. the output tile is rounded to the I/O dtype and stored once.
//
// MFMA 32x32x16 layouts (lane l, h = l / 32): A: row l % 32, k = 8h + j;
// B: column l % 32, k = 8h + j; D: column l % 32, rows 8q + 4h + i in
// register 4q + i.  Products are transposed ("swap-AB") so pixels are MFMA
// columns.  Two row permutations make every operand a single 16-byte load:
//   sigma(m) = 16*(m>>4) + 8*((m>>2)&1) + 4*((m>>3)&1) + (m&3)
// gathers the expand rows so that expand registers 8kk..8kk+7 of lane group h
// are hidden channels 16kk + 8h + 0..7 -- exactly the B fragment of the kk-th
// project K step -- and
//   tau(m) = 16*((m>>2)&1) + 4*(m>>3) + (m&3)
// gathers the project rows so that lane group h accumulates 16 consecutive
// output channels (two 16-byte stores, and 16-byte residual reads).
//
// The activation is evaluated on u / 4 (the fp16 GELU polynomial is written
// in that variable): the depth-wise output, b1 and the initial accumulators
// are pre-scaled by 1/4 and the output is multiplied by 4 -- exact powers of
// two, and every activation used here is positively homogeneous or applied
// through that change of variable.
//
// Hidden-split mode (grid.y > 1): workgroup (tile, g) runs only its range of
// chunks and writes an fp32 partial of the projected output; a second kernel
// adds the partials in group order plus b2 and the residual.
#pragma once
#include "cf_device.h"
#include "cf_kernels.h"

namespace cf {

namespace fused {

typedef float float16v __attribute__((ext_vector_type(16)));

using cf::FastDiv;
using cf::fdiv;
using cf::make_fastdiv;

struct FusedArgs {
    const uint16_t *x;
    uint16_t *y;
    const uint16_t *dw_w;
    const float *s0, *b0;
    const uint16_t *w1;
    const float *s1, *b1;
    const uint16_t *w2;
    const float *s2, *b2;
    float *partial;
    int N, H, W, E;
    uint32_t P;           // N*H*W < 2^31
    FastDiv divW, divH;
    int ntiles;
    int chunks_per_group;
    int halo_rows;        // LDS row slots for data; one more zero row follows
    int nhbuf;            // halo buffers: 2 overlaps the copy of the next slab with this one
    int dma_weights;      // weights go global->LDS untouched (no scale vectors to fold)
};

__device__ __forceinline__ u32x4 lds_ld16(const uint8_t *base, uint32_t off) {
    return *reinterpret_cast<const u32x4 *>(base + off);
}

// s_waitcnt vmcnt(n) leaving LDS/export counters alone (gfx9 encoding:
// vmcnt in bits 3:0 and 15:14, expcnt 6:4, lgkmcnt 11:8).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}
// Wait until at most n vector-memory operations of this wave are
// outstanding (n is clamped to 16; a smaller bound only waits longer).
__device__ __forceinline__ void wait_vmcnt_le(int n) {
    switch (n < 0 ? 0 : n > 16 ? 16 : n) {
    case 0: wait_vmcnt<0>(); break;
    case 1: wait_vmcnt<1>(); break;
    case 2: wait_vmcnt<2>(); break;
    case 3: wait_vmcnt<3>(); break;
    case 4: wait_vmcnt<4>(); break;
    case 5: wait_vmcnt<5>(); break;
    case 6: wait_vmcnt<6>(); break;
    case 7: wait_vmcnt<7>(); break;
    case 8: wait_vmcnt<8>(); break;
    case 9: wait_vmcnt<9>(); break;
    case 10: wait_vmcnt<10>(); break;
    case 11: wait_vmcnt<11>(); break;
    case 12: wait_vmcnt<12>(); break;
    case 13: wait_vmcnt<13>(); break;
    case 14: wait_vmcnt<14>(); break;
    case 15: wait_vmcnt<15>(); break;
    default: wait_vmcnt<16>(); break;
    }
}

// One wave-wide 16-byte global->LDS copy: lane l's 16 bytes land at
// lds_wave_base + 16 * l (a wave-uniform LDS address).  Issued as inline
// assembly: the compiler's wait-count pass cannot tell which LDS bytes a
// pending copy writes, so for its own builtin it waits for every outstanding
// copy (vmcnt 0) before each later LDS read, and a prefetch becomes a
// synchronous copy.  The pass does not see these copies; every caller waits
// for them itself (s_waitcnt vmcnt) before the destination is read or
// published by a barrier.  Vector-memory operations of a wave complete in
// issue order, so a wait the compiler places for one of its own loads stays
// correct (it can only wait longer).  M0, which holds the LDS address of the
// copy, is restored afterwards.
__device__ __forceinline__ void dma16(const void *src, uint8_t *lds_wave_base) {
    const uint32_t lds = (uint32_t)__builtin_amdgcn_readfirstlane(
        (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t *)lds_wave_base);
    uint32_t saved;
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %2\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %1, off\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved)
        : "v"(src), "s"(lds)
        : "memory");
}

// The same copy from a wave-uniform base address (held in SGPRs) plus a
// 32-bit per-lane byte offset, so that a wave keeps one VGPR per copy pattern
// instead of a 64-bit address per copy.
__device__ __forceinline__ void dma16s(const void *base, uint32_t voff, uint8_t *lds_wave_base) {
    const uint32_t lds = (uint32_t)__builtin_amdgcn_readfirstlane(
        (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t *)lds_wave_base);
    const uint64_t b = (uint64_t)(uintptr_t)base;
    // (readfirstlane returns int: go through uint32_t so that neither half is sign-extended)
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

// dma16s for the lanes set in a wave-uniform, nonzero mask (EXEC is set
// and restored inside the instruction group, so the copy needs no
// divergent branch).  The mask replaces EXEC rather than narrowing it: call
// it from wave-uniform control flow, with every lane active.
__device__ __forceinline__ void dma16m(const void *base, uint32_t voff, uint8_t *lds_wave_base, uint64_t mask) {
    const uint32_t lds = (uint32_t)__builtin_amdgcn_readfirstlane(
        (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t *)lds_wave_base);
    const uint64_t b = (uint64_t)(uintptr_t)base;
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)b);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(b >> 32));
    const uint64_t bu = ((uint64_t)hi << 32) | (uint64_t)lo;
    const uint32_t mlo = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)mask);
    const uint32_t mhi = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(mask >> 32));
    const uint64_t mu = ((uint64_t)mhi << 32) | (uint64_t)mlo;
    uint64_t saved_exec;
    uint32_t saved_m0;
    asm volatile(
        "s_mov_b64 %0, exec\n\t"
        "s_mov_b64 exec, %5\n\t"
        "s_mov_b32 %1, m0\n\t"
        "s_mov_b32 m0, %4\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %2, %3\n\t"
        "s_mov_b32 m0, %1\n\t"
        "s_mov_b64 exec, %0"
        : "=&s"(saved_exec), "=&s"(saved_m0)
        : "v"(voff), "s"(bu), "s"(lds), "s"(mu)
        : "memory");
}

// As dma16m, with the destination given as an LDS byte address rather than a
// generic pointer (no address-space conversion in the caller's loop).
__device__ __forceinline__ void dma16m_at(const void *base, uint32_t voff, uint32_t lds_addr, uint64_t mask) {
    const uint32_t lds = (uint32_t)__builtin_amdgcn_readfirstlane(lds_addr);
    const uint64_t b = (uint64_t)(uintptr_t)base;
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)b);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(b >> 32));
    const uint64_t bu = ((uint64_t)hi << 32) | (uint64_t)lo;
    const uint32_t mlo = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)mask);
    const uint32_t mhi = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(mask >> 32));
    const uint64_t mu = ((uint64_t)mhi << 32) | (uint64_t)mlo;
    uint64_t saved_exec;
    uint32_t saved_m0;
    asm volatile(
        "s_mov_b64 %0, exec\n\t"
        "s_mov_b64 exec, %5\n\t"
        "s_mov_b32 %1, m0\n\t"
        "s_mov_b32 m0, %4\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %2, %3\n\t"
        "s_mov_b32 m0, %1\n\t"
        "s_mov_b64 exec, %0"
        : "=&s"(saved_exec), "=&s"(saved_m0)
        : "v"(voff), "s"(bu), "s"(lds), "s"(mu)
        : "memory");
}

__device__ __forceinline__ float16v mfma32(const u32x4 &a, const u32x4 &b, const float16v &c, F16) {
    Pack8 pa, pb;
    pa.u = a;
    pb.u = b;
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(pa.h, pb.h, c, 0, 0, 0);
}
__device__ __forceinline__ float16v mfma32(const u32x4 &a, const u32x4 &b, const float16v &c, BF16) {
    Pack8 pa, pb;
    pa.u = a;
    pb.u = b;
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(pa.b, pb.b, c, 0, 0, 0);
}

// Scale 8 packed elements by one fp32 factor (weights with a folded norm).
template <typename T>
__device__ __forceinline__ u32x4 scale8(u32x4 v, float s) {
    u32x4 r;
#pragma unroll
    for (int q = 0; q < 4; q++)
        r[q] = T::pack2(T::lo(v[q]) * s, T::hi(v[q]) * s);
    return r;
}

__host__ __device__ constexpr int sigma_row(int m) {
    return 16 * (m >> 4) + 8 * ((m >> 2) & 1) + 4 * ((m >> 3) & 1) + (m & 3);
}
__host__ __device__ constexpr int tau_row(int m) { return 16 * ((m >> 2) & 1) + 4 * (m >> 3) + (m & 3); }

// Activation of the 1/4-scaled expand output w = u / 4, returned as
// phi(u) / 4 packed to the I/O dtype.
template <typename T, int ACT>
__device__ __forceinline__ uint32_t act_q(float a, float b) {
    if constexpr (ACT == ACT_GELU) {
        if constexpr (!T::is_bf16) {
            half2v w;
            w.x = (_Float16)a;
            w.y = (_Float16)b;
            return __builtin_bit_cast(uint32_t, gelu_pk_f16_quarter(w));
        } else {
            return T::pack2(0.25f * gelu_f32(4.0f * a), 0.25f * gelu_f32(4.0f * b));
        }
    } else if constexpr (ACT == ACT_RELU) {
        if constexpr (!T::is_bf16) {
            half2v w;
            w.x = (_Float16)a;
            w.y = (_Float16)b;
            const half2v z = {(_Float16)0.0f, (_Float16)0.0f};
            return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(w, z));
        } else {
            return T::pack2(fmaxf(a, 0.0f), fmaxf(b, 0.0f));
        }
    } else {
        return T::pack2(a, b);
    }
}

// Activation of NP packed pairs at once, written stage by stage across the
// pairs so the NP independent dependency chains interleave in the VALU.
template <typename T, int ACT, int NP>
__device__ __forceinline__ void act_pairs(const float (&a)[2 * NP], uint32_t (&out)[NP]) {
    if constexpr (ACT == ACT_GELU && !T::is_bf16) {
        const half2v c0 = splat2(GELU_Q0), c1 = splat2(GELU_Q1), c2 = splat2(GELU_Q2);
        const half2v c3 = splat2(GELU_Q3), c4 = splat2(GELU_Q4);
        const half2v half_ = splat2(0.5f), zero = splat2(0.0f), one = splat2(1.0f);
        half2v w[NP], sq[NP], q[NP];
#pragma unroll
        for (int p = 0; p < NP; p++) {
            w[p].x = (_Float16)a[2 * p];
            w[p].y = (_Float16)a[2 * p + 1];
        }
#pragma unroll
        for (int p = 0; p < NP; p++)
            sq[p] = w[p] * w[p];
#pragma unroll
        for (int p = 0; p < NP; p++)
            q[p] = __builtin_elementwise_fma(sq[p], c4, c3);
#pragma unroll
        for (int p = 0; p < NP; p++)
            q[p] = __builtin_elementwise_fma(sq[p], q[p], c2);
#pragma unroll
        for (int p = 0; p < NP; p++)
            q[p] = __builtin_elementwise_fma(sq[p], q[p], c1);
#pragma unroll
        for (int p = 0; p < NP; p++)
            q[p] = __builtin_elementwise_fma(sq[p], q[p], c0);
#pragma unroll
        for (int p = 0; p < NP; p++)
            q[p] = __builtin_elementwise_min(__builtin_elementwise_max(__builtin_elementwise_fma(w[p], q[p], half_), zero), one);
#pragma unroll
        for (int p = 0; p < NP; p++)
            out[p] = __builtin_bit_cast(uint32_t, w[p] * q[p]);
    } else {
#pragma unroll
        for (int p = 0; p < NP; p++)
            out[p] = act_q<T, ACT>(a[2 * p], a[2 * p + 1]);
    }
}

template <int C, int KS, int NWAVE, int NB, typename T, int ACT, bool RESIDENT>
struct Fused {
    static constexpr int NT = NWAVE * 64;
    static constexpr int M = NWAVE * NB * 32;   // pixels per tile
    static constexpr int PAD = KS / 2;
    static constexpr int CS = 64;               // channels per halo slab
    static constexpr int NSLAB = C / CS;
    static constexpr int KST = C / 16;          // expand K steps
    static constexpr int KSL = CS / 16;         // K steps per slab
    static constexpr int CB = C / 32;           // output channel blocks of 32
    static constexpr int W1_BYTES = KST * 1024; // expand fragments of a chunk
    static constexpr int CHUNK_BYTES = 128 * C + 128;
    static constexpr int PIECES = (8 * C + NT - 1) / NT;  // 16-byte weight pieces per thread per chunk
    static constexpr int PSTRIDE = CS * 2;      // bytes per pixel in a halo slab
    static constexpr float QS = 0.25f;          // activation-variable scale
    // staged per-channel constants: s0/4, b0/4 (fp16 or fp32), b2/4 (fp32)
    static constexpr int CST_B0 = T::is_bf16 ? 4 * C : 2 * C;
    static constexpr int CST_B2 = 2 * CST_B0;
    static constexpr int CST_BYTES = CST_B2 + 4 * C;

    // ------------------------------------------------------------------ weights
    // Chunk layout in LDS: [KST][64 lanes][16 B] W1 fragments, then
    // [CB][2][64][16 B] W2 fragments, then b1 as [h][16 floats] (scaled by QS).
    static __device__ __forceinline__ const uint16_t *w1_src(const FusedArgs &a, int r0, int ks, int lane,
                                                             int &row) {
        row = r0 + sigma_row(lane & 31);
        return a.w1 + (size_t)row * C + ks * 16 + 8 * (lane >> 5);
    }
    static __device__ __forceinline__ const uint16_t *w2_src(const FusedArgs &a, int r0, int cb, int kk, int lane,
                                                             int &row) {
        row = cb * 32 + tau_row(lane & 31);
        return a.w2 + (size_t)row * (a.E * C) + r0 + 16 * kk + 8 * (lane >> 5);
    }

    // b1 slice of chunk ch in the expand register order, scaled by QS:
    // 8 threads, 4 floats each.
    static __device__ __forceinline__ void stage_b1(const FusedArgs &a, int ch, int tid, uint8_t *buf) {
        if (tid < 8) {
            const int h = tid >> 2, t = tid & 3;
            const int r = ch * 32 + 16 * (t >> 1) + 8 * h + 4 * (t & 1);
            float4v v = a.b1 ? *reinterpret_cast<const float4v *>(a.b1 + r) : float4v{0.f, 0.f, 0.f, 0.f};
            *reinterpret_cast<float4v *>(buf + 128 * C + tid * 16) = v * QS;
        }
    }

    // Asynchronous copy of chunk ch (no scale folding): one 1 KB fragment per
    // wave instruction.
    static __device__ __forceinline__ void chunk_dma(const FusedArgs &a, int ch, int wv, int lane, uint8_t *buf) {
        const int r0 = ch * 32;
        constexpr int NFR = KST + 2 * CB;
        for (int f = wv; f < NFR; f += NWAVE) {
            int row;
            const uint16_t *src;
            if (f < KST)
                src = w1_src(a, r0, f, lane, row);
            else
                src = w2_src(a, r0, (f - KST) >> 1, (f - KST) & 1, lane, row);
            dma16(src, buf + f * 1024);
        }
    }

    // Register-staged copy of chunk ch with s1 / s2 folded into the rows.
    static __device__ __forceinline__ void chunk_load(const FusedArgs &a, int ch, int tid, u32x4 (&reg)[PIECES]) {
        const int r0 = ch * 32;
#pragma unroll
        for (int q = 0; q < PIECES; q++) {
            const int p = q * NT + tid;
            if (p >= 8 * C)
                continue;
            const int f = p >> 6, l = p & 63;
            int row;
            const uint16_t *src;
            const float *sv;
            if (f < KST) {
                src = w1_src(a, r0, f, l, row);
                sv = a.s1;
            } else {
                src = w2_src(a, r0, (f - KST) >> 1, (f - KST) & 1, l, row);
                sv = a.s2;
            }
            const u32x4 v = *reinterpret_cast<const u32x4 *>(src);
            reg[q] = sv ? scale8<T>(v, sv[row]) : v;
        }
    }
    static __device__ __forceinline__ void chunk_store(uint8_t *buf, int tid, const u32x4 (&reg)[PIECES]) {
#pragma unroll
        for (int q = 0; q < PIECES; q++) {
            const int p = q * NT + tid;
            if (p < 8 * C)
                *reinterpret_cast<u32x4 *>(buf + (size_t)p * 16) = reg[q];
        }
    }

    // Expand of one chunk of 32 hidden channels for this wave's NB pixel
    // blocks: hacc = W1_chunk D^T + b1 (b1 enters through the C operand).
    static __device__ __forceinline__ void expand(const uint8_t *buf, int lane, const u32x4 (&dfr)[KST][NB],
                                                  float16v (&hacc)[NB]) {
        const int h = lane >> 5;
        const float16v bias = *reinterpret_cast<const float16v *>(buf + 128 * C + h * 64);
#pragma unroll
        for (int ks = 0; ks < KST; ks++) {
            const u32x4 af = lds_ld16(buf, (uint32_t)((ks * 64 + lane) * 16));
#pragma unroll
            for (int b = 0; b < NB; b++)
                hacc[b] = mfma32(af, dfr[ks][b], ks == 0 ? bias : hacc[b], T{});
        }
    }

    // Activation of an expanded chunk and its projection onto the output
    // accumulators: acc += W2_chunk phi(hacc).
    static __device__ __forceinline__ void project(const uint8_t *buf, int lane, const float16v (&hacc)[NB],
                                                   float16v (&acc)[CB][NB]) {
        u32x4 hid[NB][2];
#pragma unroll
        for (int b = 0; b < NB; b++)
#pragma unroll
            for (int kk = 0; kk < 2; kk++)
#pragma unroll
                for (int p = 0; p < 4; p++)
                    hid[b][kk][p] = act_q<T, ACT>(hacc[b][8 * kk + 2 * p], hacc[b][8 * kk + 2 * p + 1]);
#pragma unroll
        for (int cb = 0; cb < CB; cb++)
#pragma unroll
            for (int kk = 0; kk < 2; kk++) {
                const u32x4 wf = lds_ld16(buf, (uint32_t)(W1_BYTES + ((cb * 2 + kk) * 64 + lane) * 16));
#pragma unroll
                for (int b = 0; b < NB; b++)
                    acc[cb][b] = mfma32(wf, hid[b][kk], acc[cb][b], T{});
            }
    }

    // ---- software-pipelined FFN over NCH resident chunks.
    // Iteration c: activation of chunk c (VALU), expand of chunk c+1 and
    // project of chunk c-1 (MFMA) -- mutually independent, so the scheduler
    // interleaves one MFMA with a run of VALU instructions -- while the LDS
    // fragments of the next iteration are fetched.
    static __device__ __forceinline__ void load_w1(const uint8_t *buf, int lane, u32x4 (&w1)[KST], float16v &bias) {
        bias = *reinterpret_cast<const float16v *>(buf + 128 * C + (lane >> 5) * 64);
#pragma unroll
        for (int ks = 0; ks < KST; ks++)
            w1[ks] = lds_ld16(buf, (uint32_t)((ks * 64 + lane) * 16));
    }
    static __device__ __forceinline__ void load_w2(const uint8_t *buf, int lane, u32x4 (&w2)[CB][2]) {
#pragma unroll
        for (int cb = 0; cb < CB; cb++)
#pragma unroll
            for (int kk = 0; kk < 2; kk++)
                w2[cb][kk] = lds_ld16(buf, (uint32_t)(W1_BYTES + ((cb * 2 + kk) * 64 + lane) * 16));
    }
    static __device__ __forceinline__ void mma_expand(const u32x4 (&w1)[KST], const float16v &bias,
                                                      const u32x4 (&dfr)[KST][NB], float16v (&hh)[NB]) {
#pragma unroll
        for (int ks = 0; ks < KST; ks++)
#pragma unroll
            for (int b = 0; b < NB; b++)
                hh[b] = mfma32(w1[ks], dfr[ks][b], ks == 0 ? bias : hh[b], T{});
    }
    static __device__ __forceinline__ void mma_project(const u32x4 (&w2)[CB][2], const u32x4 (&hid)[NB][2],
                                                       float16v (&acc)[CB][NB]) {
#pragma unroll
        for (int kk = 0; kk < 2; kk++)
#pragma unroll
            for (int cb = 0; cb < CB; cb++)
#pragma unroll
                for (int b = 0; b < NB; b++)
                    acc[cb][b] = mfma32(w2[cb][kk], hid[b][kk], acc[cb][b], T{});
    }
    static __device__ __forceinline__ void activate(const float16v (&hh)[NB], u32x4 (&hid)[NB][2]) {
        float v[NB * 16];
#pragma unroll
        for (int b = 0; b < NB; b++)
#pragma unroll
            for (int e = 0; e < 16; e++)
                v[b * 16 + e] = hh[b][e];
        uint32_t o[NB * 8];
        act_pairs<T, ACT, NB * 8>(v, o);
#pragma unroll
        for (int b = 0; b < NB; b++)
#pragma unroll
            for (int kk = 0; kk < 2; kk++)
#pragma unroll
                for (int p = 0; p < 4; p++)
                    hid[b][kk][p] = o[b * 8 + kk * 4 + p];
    }

    template <int NCH>
    static __device__ __forceinline__ void ffn_pipelined(const uint8_t *wbuf, int lane, const u32x4 (&dfr)[KST][NB],
                                                         float16v (&acc)[CB][NB]) {
        float16v hh[2][NB];
        u32x4 hid[2][NB][2];
        u32x4 w1[2][KST];
        float16v bias[2];
        u32x4 w2[2][CB][2];
        load_w1(wbuf, lane, w1[0], bias[0]);
        mma_expand(w1[0], bias[0], dfr, hh[0]);
        if constexpr (NCH > 1)
            load_w1(wbuf + CHUNK_BYTES, lane, w1[1], bias[1]);
#pragma unroll
        for (int c = 0; c < NCH; c++) {
            const int cur = c & 1, nxt = cur ^ 1;
            if (c + 2 < NCH)
                load_w1(wbuf + (size_t)(c + 2) * CHUNK_BYTES, lane, w1[cur], bias[cur]);
            load_w2(wbuf + (size_t)c * CHUNK_BYTES, lane, w2[cur]);
            activate(hh[cur], hid[cur]);
            if (c + 1 < NCH)
                mma_expand(w1[nxt], bias[nxt], dfr, hh[nxt]);
            if (c >= 1)
                mma_project(w2[nxt], hid[nxt], acc);
            // interleave: one MFMA, then a run of VALU instructions
#pragma unroll
            for (int g = 0; g < KST * NB + 2 * CB * NB; g++) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x002, 8, 0);
            }
        }
        mma_project(w2[(NCH - 1) & 1], hid[(NCH - 1) & 1], acc);
    }

    static __device__ __forceinline__ void chunk_compute(const uint8_t *buf, int lane, const u32x4 (&dfr)[KST][NB],
                                                         float16v (&acc)[CB][NB]) {
        float16v hacc[NB];
        expand(buf, lane, dfr, hacc);
        project(buf, lane, hacc, acc);
    }

    // ------------------------------------------------------------------ halo
    // LDS layout of one halo slab: [halo_rows + 1][W + 2*PAD][64 channels],
    // 128 bytes per pixel, the last row all zeros (read by taps that fall
    // outside the pixel's image).  Inside a pixel the eight 16-byte channel
    // chunks are XOR-swizzled by the LDS column (logical chunk q at
    // q ^ (col & 7)), so 8 neighbouring pixels read by 8 lanes hit 8
    // different bank groups.  The k*k*64 taps of the slab follow the halo.
    static __device__ __forceinline__ uint32_t swz(uint32_t col, uint32_t q) { return q ^ (col & 7u); }

    static __device__ __forceinline__ void issue_slab(const FusedArgs &a, uint8_t *hbuf, uint8_t *wbuf_dw,
                                                      uint32_t g_lo, int rows, int slab, int wv, int lane) {
        const int W = a.W;
        const int WP = W + 2 * PAD;
        const int64_t NH = (int64_t)a.N * a.H;
        const int per_row = W * (CS / 8);  // 16-byte chunks per row interior
        const int ipr = (per_row + 63) >> 6;
        const int total = rows * ipr;
        int r = 0, part = wv;
        while (part >= ipr) {
            part -= ipr;
            r++;
        }
        for (int j = wv; j < total; j += NWAVE) {
            const int64_t grow = (int64_t)g_lo - PAD + r;
            if (grow >= 0 && grow < NH) {
                const int ci = part * 64 + lane;
                if (ci < per_row) {
                    const int p = ci >> 3, c = ci & 7;
                    const uint32_t q = swz((uint32_t)(p + PAD), (uint32_t)c);
                    const uint16_t *src = a.x + (((size_t)grow * W + p) * C + slab * CS + q * 8);
                    dma16(src, hbuf + ((size_t)r * WP + PAD) * PSTRIDE + (size_t)part * 1024);
                }
            }
            part += NWAVE;
            while (part >= ipr) {
                part -= ipr;
                r++;
            }
        }
        constexpr int TCH = KS * KS * (CS / 8);
        for (int j = wv; j * 64 < TCH; j += NWAVE) {
            const int ci = j * 64 + lane;
            if (ci < TCH) {
                const int tap = ci >> 3, q = ci & 7;
                dma16(a.dw_w + ((size_t)tap * C + slab * CS + q * 8), wbuf_dw + j * 1024);
            }
        }
    }

    static __device__ __forceinline__ void tile_geom(const FusedArgs &a, int tile, uint32_t &p0, uint32_t &pend,
                                                     uint32_t &g_lo, int &rows) {
        p0 = (uint32_t)tile * M;
        pend = p0 + M < a.P ? p0 + M : a.P;
        g_lo = fdiv(p0, a.divW);
        const uint32_t g_hi = fdiv(pend - 1, a.divW);
        rows = (int)(g_hi - g_lo) + 1 + 2 * PAD;
    }

    static __device__ void run(const FusedArgs &a, uint8_t *smem) {
        const bool split = a.partial != nullptr;
        const int tid = threadIdx.x;
        const int lane = tid & 63, wv = tid >> 6;
        const int h = lane >> 5, m = lane & 31;
        const int W = a.W;
        const int WP = W + 2 * PAD;
        const int ch_begin = blockIdx.y * a.chunks_per_group;
        const int ch_end = ch_begin + a.chunks_per_group;
        const int NHBUF = a.nhbuf;

        const uint32_t halo_bytes = (uint32_t)(a.halo_rows + 1) * WP * PSTRIDE;
        const uint32_t dw_bytes = ((uint32_t)KS * KS * PSTRIDE + 255u) & ~255u;
        const uint32_t hbuf_bytes = ((halo_bytes + 255u) & ~255u) + dw_bytes;
        uint8_t *wbuf = smem + NHBUF * hbuf_bytes;
        // per-channel constants staged once: s0/4 and b0/4 (packed fp16 for
        // fp16 I/O, fp32 for bf16), then (b2/4) in fp32
        uint8_t *cst = wbuf + (size_t)(RESIDENT ? a.chunks_per_group : 2) * CHUNK_BYTES;
        const uint32_t zrow = (uint32_t)a.halo_rows * WP * PSTRIDE;  // byte offset of the zero row

        // Halo buffers start at zero: pad columns and the zero row are never
        // written again.
        for (uint32_t i = tid; i < NHBUF * hbuf_bytes / 16; i += NT)
            reinterpret_cast<u32x4 *>(smem)[i] = u32x4{0u, 0u, 0u, 0u};
        for (int c = tid; c < C; c += NT) {
            const float sq = (a.s0 ? a.s0[c] : 1.0f) * QS, bq = (a.b0 ? a.b0[c] : 0.0f) * QS;
            if constexpr (!T::is_bf16) {
                reinterpret_cast<_Float16 *>(cst)[c] = (_Float16)sq;
                reinterpret_cast<_Float16 *>(cst + CST_B0)[c] = (_Float16)bq;
            } else {
                reinterpret_cast<float *>(cst)[c] = sq;
                reinterpret_cast<float *>(cst + CST_B0)[c] = bq;
            }
            reinterpret_cast<float *>(cst + CST_B2)[c] = (split || !a.b2) ? 0.0f : a.b2[c] * QS;
        }
        __syncthreads();

        if constexpr (RESIDENT) {
            for (int ch = ch_begin; ch < ch_end; ch++) {
                uint8_t *cbuf = wbuf + (size_t)(ch - ch_begin) * CHUNK_BYTES;
                if (a.dma_weights) {
                    chunk_dma(a, ch, wv, lane, cbuf);
                } else {
                    u32x4 reg[PIECES];
                    chunk_load(a, ch, tid, reg);
                    chunk_store(cbuf, tid, reg);
                }
                stage_b1(a, ch, tid, cbuf);
            }
        }

        int tile = blockIdx.x;
        if (tile < a.ntiles) {
            uint32_t p0, pend, g_lo;
            int rows;
            tile_geom(a, tile, p0, pend, g_lo, rows);
            issue_slab(a, smem, smem + hbuf_bytes - dw_bytes, g_lo, rows, 0, wv, lane);
        }
        int item = 0;
        // vector-memory operations this wave issued after the copy of the
        // next halo item (the previous tile's output stores): memory
        // operations retire in order, so waiting for "at most this many
        // outstanding" waits for the copy but not for the stores
        int stores_after_copy = 0;
        for (; tile < a.ntiles; tile += gridDim.x) {
            uint32_t p0, pend, g_lo;
            int rows;
            tile_geom(a, tile, p0, pend, g_lo, rows);
            const int next_tile = tile + gridDim.x;

            // per-lane pixel bookkeeping for this tile
            uint32_t ctr[NB];    // byte offset of the pixel's own row in a slab
            uint32_t rmask[NB];  // bit i: kernel row i lies inside the pixel's image
            uint32_t pix[NB];
            bool valid[NB];
            int lcol[NB];        // LDS column of the pixel (image column + PAD)
#pragma unroll
            for (int b = 0; b < NB; b++) {
                const uint32_t s = (uint32_t)((wv * NB + b) * 32 + m);
                pix[b] = p0 + s;
                valid[b] = pix[b] < pend;
                const uint32_t gg = valid[b] ? fdiv(pix[b], a.divW) : g_lo;
                const int wc = valid[b] ? (int)(pix[b] - gg * (uint32_t)W) : 0;
                const int hh = (int)(gg - fdiv(gg, a.divH) * (uint32_t)a.H);
                lcol[b] = wc + PAD;
                ctr[b] = (gg - g_lo + PAD) * (uint32_t)WP * PSTRIDE;
                uint32_t msk = 0;
#pragma unroll
                for (int i = 0; i < KS; i++) {
                    const int hr = hh + i - PAD;
                    if (valid[b] && hr >= 0 && hr < a.H)
                        msk |= 1u << i;
                }
                rmask[b] = msk;
            }
            // byte offset of tap column j, K step ksl, within a halo row:
            // column * 128 + ((2*ksl + h) ^ (column & 7)) * 16
            uint32_t colx[NB][KSL][KS];
#pragma unroll
            for (int b = 0; b < NB; b++)
#pragma unroll
                for (int j = 0; j < KS; j++) {
                    const uint32_t col = (uint32_t)(lcol[b] - PAD + j);
                    const uint32_t base = (col << 7) | (((uint32_t)h ^ (col & 7u)) << 4);
#pragma unroll
                    for (int ksl = 0; ksl < KSL; ksl++)
                        colx[b][ksl][j] = base ^ ((uint32_t)ksl << 5);
                }

            u32x4 dfr[KST][NB];
            float16v acc[CB][NB];

#pragma unroll
            for (int slab = 0; slab < NSLAB; slab++, item++) {
                // LDS pointers are formed from the __shared__ base so that they stay
                // in the LDS address space (ds_read, not flat loads)
                uint8_t *halo = smem + ((NHBUF == 2 && (item & 1)) ? hbuf_bytes : 0u);
                const uint8_t *dww = halo + hbuf_bytes - dw_bytes;
                // this wave's copies of the item have landed ...
                if constexpr (RESIDENT && NSLAB == 1)
                    wait_vmcnt_le(stores_after_copy);
                else
                    __builtin_amdgcn_s_waitcnt(0);
                __syncthreads();  // ... and every other wave's
                if (NHBUF == 2) {
                    uint8_t *nb = smem + (((item + 1) & 1) ? hbuf_bytes : 0u);
                    if (slab + 1 < NSLAB)
                        issue_slab(a, nb, nb + hbuf_bytes - dw_bytes, g_lo, rows, slab + 1, wv, lane);
                    else if (next_tile < a.ntiles) {
                        uint32_t q0, qend, qg;
                        int qrows;
                        tile_geom(a, next_tile, q0, qend, qg, qrows);
                        issue_slab(a, nb, nb + hbuf_bytes - dw_bytes, qg, qrows, 0, wv, lane);
                    }
                }

                // ---- depth-wise conv on the VALU for the K steps of this slab
                if constexpr (!T::is_bf16) {
                    half2v accd[KSL][NB][4];
#pragma unroll
                    for (int ksl = 0; ksl < KSL; ksl++)
#pragma unroll
                        for (int b = 0; b < NB; b++)
#pragma unroll
                            for (int q = 0; q < 4; q++)
                                accd[ksl][b][q] = half2v{(_Float16)0.0f, (_Float16)0.0f};
#pragma unroll 1
                    for (int i = 0; i < KS; i++) {
                        uint32_t rowoff[NB];
#pragma unroll
                        for (int b = 0; b < NB; b++)
                            rowoff[b] = ((rmask[b] >> i) & 1u) ? ctr[b] + (uint32_t)((i - PAD) * WP * PSTRIDE) : zrow;
#pragma unroll
                        for (int ksl = 0; ksl < KSL; ksl++) {
                            Pack8 wr[KS];
#pragma unroll
                            for (int j = 0; j < KS; j++)
                                wr[j].u = lds_ld16(dww, (uint32_t)((i * KS + j) * PSTRIDE + ((2 * ksl + h) << 4)));
#pragma unroll
                            for (int b = 0; b < NB; b++)
#pragma unroll
                                for (int j = 0; j < KS; j++) {
                                    Pack8 v;
                                    v.u = lds_ld16(halo, rowoff[b] + colx[b][ksl][j]);
#pragma unroll
                                    for (int q = 0; q < 4; q++)
                                        accd[ksl][b][q] = __builtin_elementwise_fma(
                                            __builtin_bit_cast(half2v, v.w[q]), __builtin_bit_cast(half2v, wr[j].w[q]),
                                            accd[ksl][b][q]);
                                }
                        }
                        __builtin_amdgcn_sched_barrier(0);
                    }
#pragma unroll
                    for (int ksl = 0; ksl < KSL; ksl++) {
                        const int c0 = (slab * KSL + ksl) * 16 + 8 * h;
                        Pack8 sp, bp;
                        sp.u = *reinterpret_cast<const u32x4 *>(cst + 2 * c0);
                        bp.u = *reinterpret_cast<const u32x4 *>(cst + CST_B0 + 2 * c0);
#pragma unroll
                        for (int b = 0; b < NB; b++)
#pragma unroll
                            for (int q = 0; q < 4; q++)
                                dfr[slab * KSL + ksl][b][q] = __builtin_bit_cast(
                                    uint32_t, __builtin_elementwise_fma(accd[ksl][b][q], __builtin_bit_cast(half2v, sp.w[q]),
                                                                        __builtin_bit_cast(half2v, bp.w[q])));
                    }
                } else {
#pragma unroll
                    for (int ksl = 0; ksl < KSL; ksl++) {
                        const int c0 = (slab * KSL + ksl) * 16 + 8 * h;
                        float accd[NB][8];
#pragma unroll
                        for (int b = 0; b < NB; b++)
#pragma unroll
                            for (int e = 0; e < 8; e++)
                                accd[b][e] = 0.0f;
#pragma unroll 1
                        for (int i = 0; i < KS; i++) {
                            uint32_t rowoff[NB];
#pragma unroll
                            for (int b = 0; b < NB; b++)
                                rowoff[b] = ((rmask[b] >> i) & 1u) ? ctr[b] + (uint32_t)((i - PAD) * WP * PSTRIDE) : zrow;
#pragma unroll
                            for (int j = 0; j < KS; j++) {
                                Pack8 wr;
                                wr.u = lds_ld16(dww, (uint32_t)((i * KS + j) * PSTRIDE + ((2 * ksl + h) << 4)));
#pragma unroll
                                for (int b = 0; b < NB; b++) {
                                    Pack8 v;
                                    v.u = lds_ld16(halo, rowoff[b] + colx[b][ksl][j]);
#pragma unroll
                                    for (int q = 0; q < 4; q++) {
                                        accd[b][2 * q] = fmaf(T::lo(v.w[q]), T::lo(wr.w[q]), accd[b][2 * q]);
                                        accd[b][2 * q + 1] = fmaf(T::hi(v.w[q]), T::hi(wr.w[q]), accd[b][2 * q + 1]);
                                    }
                                }
                            }
                        }
                        const float *sq = reinterpret_cast<const float *>(cst) + c0;
                        const float *bq = reinterpret_cast<const float *>(cst + CST_B0) + c0;
#pragma unroll
                        for (int b = 0; b < NB; b++)
#pragma unroll
                            for (int q = 0; q < 4; q++)
                                dfr[slab * KSL + ksl][b][q] =
                                    T::pack2(fmaf(accd[b][2 * q], sq[2 * q], bq[2 * q]),
                                             fmaf(accd[b][2 * q + 1], sq[2 * q + 1], bq[2 * q + 1]));
                    }
                }

                // ---- residual shortcut from the halo centre: acc = x / 4 + b2 / 4
                if constexpr (NSLAB == 1) {
#pragma unroll
                    for (int cb = 0; cb < CB; cb++) {
                        const int cc = cb * 32 + 16 * h;
                        const float16v bias = *reinterpret_cast<const float16v *>(cst + CST_B2 + 4 * cc);
#pragma unroll
                        for (int b = 0; b < NB; b++) {
                            if (split) {
                                acc[cb][b] = bias;
                                continue;
                            }
                            const uint32_t q0 = (uint32_t)(4 * cb + 2 * h);
                            const uint32_t col = (uint32_t)lcol[b];
                            Pack8 v0, v1;
                            v0.u = lds_ld16(halo, ctr[b] + (col << 7) + (swz(col, q0) << 4));
                            v1.u = lds_ld16(halo, ctr[b] + (col << 7) + (swz(col, q0 + 1) << 4));
                            float16v t;
#pragma unroll
                            for (int q = 0; q < 4; q++) {
                                t[2 * q] = fmaf(T::lo(v0.w[q]), QS, bias[2 * q]);
                                t[2 * q + 1] = fmaf(T::hi(v0.w[q]), QS, bias[2 * q + 1]);
                                t[8 + 2 * q] = fmaf(T::lo(v1.w[q]), QS, bias[8 + 2 * q]);
                                t[8 + 2 * q + 1] = fmaf(T::hi(v1.w[q]), QS, bias[8 + 2 * q + 1]);
                            }
                            acc[cb][b] = t;
                        }
                    }
                }

                if (NHBUF == 1) {
                    // the single buffer is free once every wave has read it
                    __syncthreads();
                    if (slab + 1 < NSLAB)
                        issue_slab(a, smem, smem + hbuf_bytes - dw_bytes, g_lo, rows, slab + 1, wv, lane);
                    else if (next_tile < a.ntiles) {
                        uint32_t q0, qend, qg;
                        int qrows;
                        tile_geom(a, next_tile, q0, qend, qg, qrows);
                        issue_slab(a, smem, smem + hbuf_bytes - dw_bytes, qg, qrows, 0, wv, lane);
                    }
                }
            }

            if constexpr (NSLAB > 1) {
                // ---- residual shortcut from x (just copied through L2 for the halo)
#pragma unroll
                for (int cb = 0; cb < CB; cb++) {
                    const int cc = cb * 32 + 16 * h;
#pragma unroll
                    for (int b = 0; b < NB; b++) {
                        float16v t;
                        if (split || !valid[b]) {
#pragma unroll
                            for (int e = 0; e < 16; e++)
                                t[e] = 0.0f;
                        } else {
                            Pack8 v0, v1;
                            v0.u = *reinterpret_cast<const u32x4 *>(a.x + (size_t)pix[b] * C + cc);
                            v1.u = *reinterpret_cast<const u32x4 *>(a.x + (size_t)pix[b] * C + cc + 8);
#pragma unroll
                            for (int q = 0; q < 4; q++) {
                                t[2 * q] = T::lo(v0.w[q]);
                                t[2 * q + 1] = T::hi(v0.w[q]);
                                t[8 + 2 * q] = T::lo(v1.w[q]);
                                t[8 + 2 * q + 1] = T::hi(v1.w[q]);
                            }
                            const float16v bias = *reinterpret_cast<const float16v *>(cst + CST_B2 + 4 * cc);
#pragma unroll
                            for (int e = 0; e < 16; e++)
                                t[e] = fmaf(t[e], QS, bias[e]);
                        }
                        acc[cb][b] = t;
                    }
                }
            }

            // ---- FFN: loop over hidden chunks (eq. e:ffn-eff)
            if constexpr (RESIDENT) {
              if (ch_end - ch_begin == 8) {
                ffn_pipelined<8>(wbuf, lane, dfr, acc);
              } else {
                // Software pipeline: the expand MFMAs of chunk c+1 are issued
                // before the activation of chunk c, so the matrix cores work
                // while the VALU evaluates phi.
                float16v hA[NB], hB[NB];
                int ch = ch_begin;
                expand(wbuf, lane, dfr, hA);
                for (; ch + 2 <= ch_end; ch += 2) {
                    const uint8_t *b0p = wbuf + (size_t)(ch - ch_begin) * CHUNK_BYTES;
                    expand(b0p + CHUNK_BYTES, lane, dfr, hB);
                    project(b0p, lane, hA, acc);
                    if (ch + 2 < ch_end)
                        expand(b0p + 2 * CHUNK_BYTES, lane, dfr, hA);
                    project(b0p + CHUNK_BYTES, lane, hB, acc);
                }
                if (ch < ch_end)
                    project(wbuf + (size_t)(ch - ch_begin) * CHUNK_BYTES, lane, hA, acc);
              }
            } else {
                if (a.dma_weights) {
                    chunk_dma(a, ch_begin, wv, lane, wbuf);
                    stage_b1(a, ch_begin, tid, wbuf);
                    for (int ch = ch_begin; ch < ch_end; ch++) {
                        const int bi = (ch - ch_begin) & 1;
                        __builtin_amdgcn_s_waitcnt(0);
                        __syncthreads();
                        if (ch + 1 < ch_end) {
                            uint8_t *nbuf = wbuf + (size_t)(bi ^ 1) * CHUNK_BYTES;
                            chunk_dma(a, ch + 1, wv, lane, nbuf);
                            stage_b1(a, ch + 1, tid, nbuf);
                        }
                        chunk_compute(wbuf + (size_t)bi * CHUNK_BYTES, lane, dfr, acc);
                    }
                } else {
                    {
                        u32x4 reg[PIECES];
                        chunk_load(a, ch_begin, tid, reg);
                        chunk_store(wbuf, tid, reg);
                        stage_b1(a, ch_begin, tid, wbuf);
                    }
                    for (int ch = ch_begin; ch < ch_end; ch++) {
                        const int bi = (ch - ch_begin) & 1;
                        __syncthreads();
                        const bool more = ch + 1 < ch_end;
                        u32x4 reg[PIECES];
                        if (more)
                            chunk_load(a, ch + 1, tid, reg);
                        chunk_compute(wbuf + (size_t)bi * CHUNK_BYTES, lane, dfr, acc);
                        if (more) {
                            chunk_store(wbuf + (size_t)(bi ^ 1) * CHUNK_BYTES, tid, reg);
                            stage_b1(a, ch + 1, tid, wbuf + (size_t)(bi ^ 1) * CHUNK_BYTES);
                        }
                    }
                }
                __syncthreads();  // chunk buffers are rewritten for the next tile
            }

            // ---- epilogue: y = 4 * acc, one store of the output tile
            stores_after_copy = 0;
#pragma unroll
            for (int b = 0; b < NB; b++) {
                // wave-uniform count; an under-count only makes the wait stricter
                if (__builtin_amdgcn_read_exec() && __ballot(valid[b]))
                    stores_after_copy += CB * (split ? 4 : 2);
                if (!valid[b])
                    continue;
#pragma unroll
                for (int cb = 0; cb < CB; cb++) {
                    const int cc = cb * 32 + 16 * h;
                    if (split) {
                        float4v *dst =
                            reinterpret_cast<float4v *>(a.partial + ((size_t)blockIdx.y * a.P + pix[b]) * C + cc);
#pragma unroll
                        for (int q = 0; q < 4; q++)
                            dst[q] = float4v{acc[cb][b][4 * q], acc[cb][b][4 * q + 1], acc[cb][b][4 * q + 2],
                                             acc[cb][b][4 * q + 3]} *
                                     4.0f;
                    } else {
                        u32x4 o0, o1;
#pragma unroll
                        for (int q = 0; q < 4; q++) {
                            o0[q] = T::pack2(4.0f * acc[cb][b][2 * q], 4.0f * acc[cb][b][2 * q + 1]);
                            o1[q] = T::pack2(4.0f * acc[cb][b][8 + 2 * q], 4.0f * acc[cb][b][8 + 2 * q + 1]);
                        }
                        u32x4 *dst = reinterpret_cast<u32x4 *>(a.y + (size_t)pix[b] * C + cc);
                        dst[0] = o0;
                        dst[1] = o1;
                    }
                }
            }
        }
        __builtin_amdgcn_s_waitcnt(0);
    }
};

template <int C, int KS, int NWAVE, int NB, typename T, int ACT, bool RESIDENT>
__global__ __launch_bounds__(NWAVE * 64, 1) void fused_block_kernel(FusedArgs a) {
    extern __shared__ __attribute__((aligned(256))) uint8_t smem[];
    Fused<C, KS, NWAVE, NB, T, ACT, RESIDENT>::run(a, smem);
}

// ---------------------------------------------------------------------------
// Host side: tile configuration per channel count.
struct Cfg {
    int nwave;
    int nb;
    bool resident;
};

constexpr Cfg cfg_for(int C) {
    return C == 64 ? Cfg{8, 1, true} : C == 128 ? Cfg{8, 1, false} : C == 256 ? Cfg{4, 1, false} : Cfg{4, 1, false};
}

inline int tile_pixels(int C) { return cfg_for(C).nwave * cfg_for(C).nb * 32; }

inline int halo_rows_for(int M, int k, int W, int64_t P) {
    int64_t span = (M - 1) / W + 2;
    const int64_t nrows_total = (P + W - 1) / W;
    if (span > nrows_total)
        span = nrows_total;
    return (int)span + 2 * (k / 2);
}

inline size_t lds_bytes_for(int C, int k, int W, int E, int64_t P, int groups, bool resident, int nhbuf,
                            bool bf16) {
    const int pad = k / 2;
    const int halo_rows = halo_rows_for(tile_pixels(C), k, W, P);
    const size_t halo = (size_t)(halo_rows + 1) * (W + 2 * pad) * 128;
    const size_t dw = ((size_t)k * k * 128 + 255) & ~(size_t)255;
    const size_t hbuf = ((halo + 255) & ~(size_t)255) + dw;
    const int chunks = E * C / 32 / groups;
    const size_t wb = (size_t)(resident ? chunks : 2) * (128 * C + 128);
    return nhbuf * hbuf + wb + (bf16 ? 12 : 8) * (size_t)C;
}

template <int C, int KS, typename T, int ACT>
hipError_t launch_t(const FusedArgs &a0, int groups, hipStream_t st) {
    constexpr Cfg cfgc = cfg_for(C);
    constexpr int NWAVE = cfgc.nwave, NB = cfgc.nb;
    FusedArgs a = a0;
    const int M = NWAVE * NB * 32;
    const int chunks = a.E * C / 32;
    const size_t lds_res = lds_bytes_for(C, KS, a.W, a.E, a.P, groups, true, 1, T::is_bf16);
    const bool resident = cfgc.resident && lds_res <= 160 * 1024;
    size_t lds = resident ? lds_res : lds_bytes_for(C, KS, a.W, a.E, a.P, groups, false, 1, T::is_bf16);
    a.nhbuf = 1;
    if (C > 64) {
        const size_t lds2 = lds_bytes_for(C, KS, a.W, a.E, a.P, groups, resident, 2, T::is_bf16);
        if (lds2 <= 160 * 1024) {
            lds = lds2;
            a.nhbuf = 2;
        }
    }
    if (lds > 160 * 1024)
        return hipErrorInvalidConfiguration;
    a.ntiles = (int)((a.P + M - 1) / M);
    a.chunks_per_group = chunks / groups;
    a.halo_rows = halo_rows_for(M, KS, a.W, a.P);
    a.divW = make_fastdiv((uint32_t)a.W);
    a.divH = make_fastdiv((uint32_t)a.H);
    a.dma_weights = (a.s1 == nullptr && a.s2 == nullptr) ? 1 : 0;
    const int cus = device_cu_count();
    int gx = a.ntiles < cus ? a.ntiles : cus;
    if (groups > 1)
        gx = a.ntiles;  // one tile per workgroup; the groups fill the chip
    dim3 grid(gx, groups);
    hipError_t e;
    if constexpr (cfgc.resident) {
        if (resident) {
            auto kfn = fused_block_kernel<C, KS, NWAVE, NB, T, ACT, true>;
            e = allow_full_lds((const void *)kfn);
            if (e != hipSuccess)
                return e;
            hipLaunchKernelGGL(kfn, grid, dim3(NWAVE * 64), lds, st, a);
            return hipGetLastError();
        }
    }
    auto kfn = fused_block_kernel<C, KS, NWAVE, NB, T, ACT, false>;
    e = allow_full_lds((const void *)kfn);
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(kfn, grid, dim3(NWAVE * 64), lds, st, a);
    return hipGetLastError();
}

template <int C, typename T, int ACT>
hipError_t launch_k(const FusedArgs &a, int k, int groups, hipStream_t st) {
    switch (k) {
    case 1: return launch_t<C, 1, T, ACT>(a, groups, st);
    case 3: return launch_t<C, 3, T, ACT>(a, groups, st);
    case 5: return launch_t<C, 5, T, ACT>(a, groups, st);
    case 7: return launch_t<C, 7, T, ACT>(a, groups, st);
    default: return hipErrorInvalidValue;
    }
}

// One instantiation unit per (channel count, dtype): every k and activation.
template <int C, typename T>
hipError_t launch_ct(const FusedArgs &a, int k, int act, int groups, hipStream_t st) {
    switch (act) {
    case ACT_GELU: return launch_k<C, T, ACT_GELU>(a, k, groups, st);
    case ACT_RELU: return launch_k<C, T, ACT_RELU>(a, k, groups, st);
    case ACT_NONE: return launch_k<C, T, ACT_NONE>(a, k, groups, st);
    default: return hipErrorInvalidValue;
    }
}

#define CF_FUSED_UNITS(X) X(64, F16) X(64, BF16) X(128, F16) X(128, BF16) X(256, F16) X(256, BF16) X(512, F16) X(512, BF16)
#define CF_DECL_UNIT(C, T) hipError_t launch_c##C##_##T(const FusedArgs &a, int k, int act, int groups, hipStream_t st);
CF_FUSED_UNITS(CF_DECL_UNIT)

}  // namespace fused
}  // namespace cf
