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

__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// One wave accumulates acc[MB][NB] (MB row blocks x NB col blocks of 16) over
// the k-steps (32 wide) ks = ks0 + j*stride + u, u < U, while ks < ks_end.
// ap[rb] / bp[cb] already point at this lane's row / col and k offset.
template <int MB, int NB, int U>
__device__ __forceinline__ void mma_ksteps(f32x4 (&acc)[MB][NB], const uint16_t* const (&ap)[MB],
                                           const uint16_t* const (&bp)[NB], int ks0, int ks_end,
                                           int stride) {
    for (int ks = ks0; ks < ks_end; ks += stride) {
        u32x4 a[U][MB], b[U][NB];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (ks + u < ks_end) {
#pragma unroll
                for (int cb = 0; cb < NB; ++cb) b[u][cb] = ld16(bp[cb] + (size_t)(ks + u) * 32);
#pragma unroll
                for (int rb = 0; rb < MB; ++rb) a[u][rb] = ld16(ap[rb] + (size_t)(ks + u) * 32);
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (ks + u < ks_end) {
#pragma unroll
                for (int rb = 0; rb < MB; ++rb)
#pragma unroll
                    for (int cb = 0; cb < NB; ++cb) acc[rb][cb] = mfma(a[u][rb], b[u][cb], acc[rb][cb]);
            }
        }
    }
}

// Deterministic reduction of the 8 waves' accumulators of one MT x NT tile
// (MT = 16 MB, NT = 16 NB) through LDS: (w0+w4)+(w2+w6) + (w1+w5)+(w3+w7).
// On return red[r * (NT + 4) + c] holds the tile sum for every thread.
// red must hold 4 * MT * (NT + 4) floats.
template <int MB, int NB>
__device__ __forceinline__ void reduce_waves(f32x4 (&acc)[MB][NB], float* red) {
    constexpr int NT = NB * 16, MT = MB * 16, LD = NT + 4, REG = MT * LD;
    const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
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
