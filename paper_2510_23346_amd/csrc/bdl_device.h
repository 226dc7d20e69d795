// Internal device helpers of the BD-LoRA shard kernels (gfx950, wave64).
//
// Matrix-core primitive: v_mfma_f32_16x16x32_bf16.  Lane l of a wave holds
//   A operand: row (l % 16), 8 consecutive k starting at 8 * (l / 16)
//   B operand: col (l % 16), the same 8 k
//   C/D      : col (l % 16), rows 4 * (l / 16) + i, i = 0..3
// Both operands are read straight from row-major, K-contiguous memory
// (activations [rows x K], nn.Linear weights [cols x K], transposed LoRA
// factors), one 16-byte load per lane per 16x32 block.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "bdl_launch.h"

namespace bdl {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// word 3 of a raw buffer resource on gfx950 (32-bit untyped data)
constexpr int kRawBufferWord3 = 0x00020000;

constexpr int kWaves = 8;                 // waves per workgroup (split K)
constexpr int kThreads = kWaves * 64;

__device__ __forceinline__ u32x4 ld16(const uint16_t* p) {
    return *reinterpret_cast<const u32x4*>(p);
}

__device__ __forceinline__ f32x4 mfma(u32x4 a, u32x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// fp32 -> bf16 bits, round to nearest, ties to even (finite inputs; NaN kept NaN)
__device__ __forceinline__ uint16_t f2bf(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return (uint16_t)((u >> 16) | 0x40);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// wave index as a scalar (uniform) value
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// MFMA fragment layout.  A K-contiguous matrix with rows padded to a
// multiple of 16 is stored as 1 KB fragments, fragment (rb, ks) holding the
// operand of one 16-row block for one 32-wide k-step exactly as the 64 lanes
// load it: element [(rb * KS + ks) * 512 + lane * 8 + i] is
// M[16 rb + lane % 16][32 ks + 8 (lane / 16) + i].  Weights, packed
// activations and the pool's A^T factors use it, so every operand load of a
// wave reads 1 KB of contiguous memory.
constexpr int kFrag = 512;                  // elements per fragment

__device__ __forceinline__ size_t frag_index(int rb, int ks, int KS) {
    return ((size_t)rb * KS + ks) * kFrag;
}

// Wave-level K loop over the contiguous k-step range [k0, k0 + n), n >= 1.
// ap[rb] / bp[cb] point at this lane's element of k-step 0; consecutive
// k-steps are sa / sb elements apart.  D stages of loads stay in flight: the
// loads of k-step i + D are issued right after the MFMAs of k-step i.  Load
// addresses are clamped to the last k-step, so the steady-state loop issues
// the same loads every iteration and each load's only consumer is the next
// iteration (the compiler cannot sink it next to its use); the last n % D
// k-steps are consumed after the loop.
template <int MB, int NB, int D>
__device__ __forceinline__ void mma_range(f32x4 (&acc)[MB][NB], const uint16_t* const (&ap)[MB],
                                          const uint16_t* const (&bp)[NB], int k0, int n, int sa,
                                          int sb) {
    u32x4 a[D][MB], b[D][NB];
    const int last = k0 + n - 1;
    auto load = [&](int d, int ks) {
#pragma unroll
        for (int cb = 0; cb < NB; ++cb) b[d][cb] = ld16(bp[cb] + (size_t)ks * sb);
#pragma unroll
        for (int rb = 0; rb < MB; ++rb) a[d][rb] = ld16(ap[rb] + (size_t)ks * sa);
    };
    auto comp = [&](int d) {
#pragma unroll
        for (int rb = 0; rb < MB; ++rb)
#pragma unroll
            for (int cb = 0; cb < NB; ++cb) acc[rb][cb] = mfma(a[d][rb], b[d][cb], acc[rb][cb]);
    };
#pragma unroll
    for (int d = 0; d < D; ++d) load(d, min(k0 + d, last));
    int i = 0;
    for (; i + D <= n; i += D) {
#pragma unroll
        for (int d = 0; d < D; ++d) {
            comp(d);
            load(d, min(k0 + i + d + D, last));
        }
    }
    const int rem = n - i;
#pragma unroll
    for (int d = 0; d < D; ++d)
        if (d < rem) comp(d);
}

// INT4 base weights.  One 32-bit word per lane and k-step holds the 8 values
// of the lane's B operand as nibbles q + 8, value i in bits 4 (i/2) + 16 (i%2).
// Each nibble u becomes the bf16 number 128 + u (exponent of 128, u in the low
// mantissa bits), which is exact; an extra MFMA against -136 removes the
// offset, so the matrix cores see exactly sum_k x_k q_k for the k-step.  The
// group scale is applied in fp32 to that k-step's product.
constexpr int kInt4Group = 4;                 // k-steps per scale group (128 inputs)
constexpr int kInt4FragBytes = 256;           // one k-step of one 16-column block

__device__ __forceinline__ u32x4 unpack_int4(uint32_t w) {
    return u32x4{(w & 0x000F000Fu) | 0x43004300u, ((w >> 4) & 0x000F000Fu) | 0x43004300u,
                 ((w >> 8) & 0x000F000Fu) | 0x43004300u, ((w >> 12) & 0x000F000Fu) | 0x43004300u};
}

__device__ __forceinline__ u32x4 int4_offset_operand() {
    return u32x4{0xC308C308u, 0xC308C308u, 0xC308C308u, 0xC308C308u};   // bf16 -136 x 8
}

// acc[rb][cb] += s_cb * (x_rb . q_cb) for one k-step: xa = activation
// fragments, q[cb] = the INT4 words, sc[cb] = bf16 scale bits (low half).
template <int MB, int NB>
__device__ __forceinline__ void mma_int4_kstep(f32x4 (&acc)[MB][NB], const u32x4 (&xa)[MB], const uint32_t (&q)[NB],
                                               const uint32_t (&sc)[NB]) {
    const u32x4 off = int4_offset_operand();
    const f32x4 zero = f32x4{0.f, 0.f, 0.f, 0.f};
    u32x4 w[NB];
    float s[NB];
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) {
        w[cb] = unpack_int4(q[cb]);
        s[cb] = __uint_as_float(sc[cb] << 16);
    }
#pragma unroll
    for (int rb = 0; rb < MB; ++rb) {
        const f32x4 corr = mfma(xa[rb], off, zero);
#pragma unroll
        for (int cb = 0; cb < NB; ++cb) {
            const f32x4 t = mfma(xa[rb], w[cb], corr);
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[rb][cb][i] = fmaf(s[cb], t[i], acc[rb][cb][i]);
        }
    }
}

// mma_range for an INT4 B operand: wq[cb] points at this lane's word of
// k-step 0 of block cb (k-steps kInt4FragBytes apart), ws[cb] at the block's
// scale of group 0 for this lane's column (groups 16 entries apart).
template <int MB, int NB, int D>
__device__ __forceinline__ void mma_range_int4(f32x4 (&acc)[MB][NB], const uint16_t* const (&ap)[MB],
                                               const char* const (&wq)[NB], const uint16_t* const (&ws)[NB],
                                               int k0, int n) {
    u32x4 a[D][MB];
    uint32_t q[D][NB], sc[D][NB];
    const int last = k0 + n - 1;
    auto load = [&](int d, int ks) {
#pragma unroll
        for (int cb = 0; cb < NB; ++cb) {
            q[d][cb] = *reinterpret_cast<const uint32_t*>(wq[cb] + (size_t)ks * kInt4FragBytes);
            sc[d][cb] = ws[cb][(ks / kInt4Group) * 16];
        }
#pragma unroll
        for (int rb = 0; rb < MB; ++rb) a[d][rb] = ld16(ap[rb] + (size_t)ks * kFrag);
    };
#pragma unroll
    for (int d = 0; d < D; ++d) load(d, min(k0 + d, last));
    int i = 0;
    for (; i + D <= n; i += D) {
#pragma unroll
        for (int d = 0; d < D; ++d) {
            mma_int4_kstep<MB, NB>(acc, a[d], q[d], sc[d]);
            load(d, min(k0 + i + d + D, last));
        }
    }
    const int rem = n - i;
#pragma unroll
    for (int d = 0; d < D; ++d)
        if (d < rem) mma_int4_kstep<MB, NB>(acc, a[d], q[d], sc[d]);
}

// minimum / bitwise or over the 64 lanes of a wave, as a uniform value
__device__ __forceinline__ int wave_min(int v) {
    constexpr int kMax = 0x7fffffff;
    v = min(v, __builtin_amdgcn_update_dpp(kMax, v, 0x111, 0xf, 0xf, false));   // row_shr:1
    v = min(v, __builtin_amdgcn_update_dpp(kMax, v, 0x112, 0xf, 0xf, false));   // row_shr:2
    v = min(v, __builtin_amdgcn_update_dpp(kMax, v, 0x114, 0xf, 0xf, false));   // row_shr:4
    v = min(v, __builtin_amdgcn_update_dpp(kMax, v, 0x118, 0xf, 0xf, false));   // row_shr:8
    v = min(v, __builtin_amdgcn_update_dpp(kMax, v, 0x142, 0xa, 0xf, false));   // row_bcast:15
    v = min(v, __builtin_amdgcn_update_dpp(kMax, v, 0x143, 0xc, 0xf, false));   // row_bcast:31
    return __builtin_amdgcn_readlane(v, 63);
}

__device__ __forceinline__ unsigned wave_or(unsigned v) {
    v |= (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xf, 0xf, false);
    v |= (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xf, 0xf, false);
    v |= (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xf, 0xf, false);
    v |= (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xf, 0xf, false);
    v |= (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xa, 0xf, false);
    v |= (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xc, 0xf, false);
    return (unsigned)__builtin_amdgcn_readlane((int)v, 63);
}

// Contiguous k-step range of wave w when KS k-steps are split over kWaves.
__device__ __forceinline__ void wave_krange(int KS, int w, int* k0, int* n) {
    const int q = KS / kWaves, r = KS - q * kWaves;
    *k0 = w * q + min(w, r);
    *n = q + (w < r ? 1 : 0);
}

// Deterministic reduction of the 8 waves' accumulators of one MT x NT tile
// (MT = 16 MB, NT = 16 NB) through LDS: (w0+w4)+(w2+w6) + (w1+w5)+(w3+w7).
// On return red[r * (NT + 4) + c] holds the tile sum for every thread.
// red must hold 4 * MT * (NT + 4) floats.
template <int MB, int NB>
__device__ __forceinline__ void reduce_waves(f32x4 (&acc)[MB][NB], float* red) {
    constexpr int NT = NB * 16, MT = MB * 16, LD = NT + 4, REG = MT * LD;
    const int w = wave_id(), l = threadIdx.x & 63;
    auto put = [&](float* dst) {
#pragma unroll
        for (int rb = 0; rb < MB; ++rb)
#pragma unroll
            for (int cb = 0; cb < NB; ++cb)
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    dst[(rb * 16 + 4 * (l >> 4) + i) * LD + cb * 16 + (l & 15)] = acc[rb][cb][i];
    };
    auto add = [&](const float* src) {
#pragma unroll
        for (int rb = 0; rb < MB; ++rb)
#pragma unroll
            for (int cb = 0; cb < NB; ++cb)
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    acc[rb][cb][i] += src[(rb * 16 + 4 * (l >> 4) + i) * LD + cb * 16 + (l & 15)];
    };
    if (w >= 4) put(red + (w - 4) * REG);
    __syncthreads();
    if (w < 4) add(red + w * REG);
    __syncthreads();
    if (w >= 2 && w < 4) put(red + (w - 2) * REG);
    __syncthreads();
    if (w < 2) add(red + w * REG);
    __syncthreads();
    if (w == 1) put(red);
    __syncthreads();
    if (w == 0) {
        add(red);
        put(red);
    }
    __syncthreads();
}

}  // namespace bdl
