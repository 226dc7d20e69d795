// Decode path (batches of at most kDecodeMaxT tokens): two launches after
// the prep launch.
//
//  dec_main_kernel -- one grid holding two kinds of work items, all of about
//                     the same size so the 256 CUs stay evenly loaded:
//                     * shrink items: Zp[s] = scale * X_rows A over the s-th K
//                       chunk, for one adapter group and up to 64 rank
//                       columns (Alg. 1 / Alg. 2 step "Z <- X A");
//                     * base items: Yp[s] = X W_s^T over the s-th K chunk of a
//                       64-column tile (step "Y <- X W").
//                     Items with no work (past the batch's shrink items) exit
//                     at once.  The 8 waves of an item split its columns in
//                     two halves and its k-steps in four quarters, and reduce
//                     the quarters through LDS in a fixed order.
//  dec_epi_kernel  -- out[t, n] = sum_s Yp[s][t][n]
//                                 + sum_j (sum_s Zp[s][t][j]) B^T[n][j]
//                     (steps "Y_adapter <- Z B" and "Y <- Y + Y_adapter"),
//                     in fp32, one bf16 store per output.
#include "bdl_device.h"

namespace bdl {

constexpr int kDecStages = 2;

// Eight waves as 2 column halves x 4 K-quarters: wave w owns column blocks
// 2 (w & 1) and 2 (w & 1) + 1 of the item's four, over the (w >> 1)-th
// quarter of its k-steps.  The three upper quarters hand their accumulators
// to the first through LDS (one barrier); the first-quarter waves then hold
// the item's result in the MFMA output layout.
template <int MB>
__device__ __forceinline__ void item_tile(f32x4 (&acc)[MB][2], const uint16_t* const (&ap)[MB],
                                          const uint16_t* const (&bp)[2], int kb, int ke, float* red) {
    constexpr int MT = MB * 16, LD = 36, REG = MT * LD;
    const int w = wave_id(), l = threadIdx.x & 63, cg = w & 1, kq = w >> 1;
#pragma unroll
    for (int rb = 0; rb < MB; ++rb) acc[rb][0] = acc[rb][1] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int n = ke - kb, q = n >> 2, r = n & 3;
    const int k0 = kb + kq * q + min(kq, r), nk = q + (kq < r ? 1 : 0);
    if (nk > 0) mma_range<MB, 2, kDecStages>(acc, ap, bp, k0, nk, kFrag, kFrag);
    if (kq > 0) {
        float* dst = red + ((kq - 1) * 2 + cg) * REG;
#pragma unroll
        for (int rb = 0; rb < MB; ++rb)
#pragma unroll
            for (int cb = 0; cb < 2; ++cb)
#pragma unroll
                for (int i = 0; i < 4; ++i) dst[(rb * 16 + 4 * (l >> 4) + i) * LD + cb * 16 + (l & 15)] = acc[rb][cb][i];
    }
    __syncthreads();
    if (kq == 0) {
#pragma unroll
        for (int j = 0; j < 3; ++j) {
            const float* src = red + (j * 2 + cg) * REG;
#pragma unroll
            for (int rb = 0; rb < MB; ++rb)
#pragma unroll
                for (int cb = 0; cb < 2; ++cb)
#pragma unroll
                    for (int i = 0; i < 4; ++i) acc[rb][cb][i] += src[(rb * 16 + 4 * (l >> 4) + i) * LD + cb * 16 + (l & 15)];
        }
    }
}

template <int MB>
__global__ __launch_bounds__(kThreads) void dec_main_kernel(DecArgs a) {
    constexpr int MT = MB * 16, NT = 64, LDR = 36;
    __shared__ float red[6 * (MT > 16 ? MT : 16) * LDR];
    const int w = wave_id(), l = threadIdx.x & 63, lr = l & 15, cg = w & 1, kq = w >> 1;
    int b = blockIdx.x;

    if (b < a.shrink_slots) {
        // ---- shrink item: 16 token rows of one adapter group x 64 A^T rows
        int p = 0;
        while (p + 1 < a.n_proj && b >= a.p[p + 1].shrink_base) ++p;
        const DecProj& P = a.p[p];
        const int local = b - P.shrink_base;
        const int item = local / (P.cchunks * P.ks);
        const int rem = local - item * (P.cchunks * P.ks);
        const int cc = rem / P.ks, s = rem - cc * P.ks;
        const int n_items = a.meta[1];
        if (item >= n_items) return;
        const int4 it = a.items[item];
        const int slot = it.x, nrows = it.z, r8s = it.w;
        const int ncols = P.n_slices * r8s;
        const int c0 = cc * NT;
        if (c0 >= ncols) return;
        const float sc = a.scale[slot];
        const int* prow = a.perm + it.y;
        const int KS = P.K >> 5;
        const int nblk = (ncols + 15) >> 4;
        const uint16_t* abase = a.pool + (size_t)slot * a.slot_stride + P.a_off;
        const uint16_t* ap[1];
        const uint16_t* bp[2];
        {
            const int t = prow[min(lr, nrows - 1)];
            ap[0] = P.Xp + frag_index(t >> 4, 0, KS) + ((t & 15) + 16 * (l >> 4)) * 8;
        }
#pragma unroll
        for (int cb = 0; cb < 2; ++cb)
            bp[cb] = abase + frag_index(min((c0 >> 4) + 2 * cg + cb, nblk - 1), 0, KS) + l * 8;
        f32x4 acc[1][2];
        const int kb = s * P.kchunk;
        item_tile<1>(acc, ap, bp, kb, min(KS, kb + P.kchunk), red);
        if (kq == 0) {
            float* zdst = P.Zp + (size_t)s * kDecodeMaxT * P.zs;
#pragma unroll
            for (int cb = 0; cb < 2; ++cb) {
                const int cgl = c0 + cg * 32 + cb * 16 + lr;
                if (cgl < ncols) {
                    const int sig = cgl / r8s, j = cgl - sig * r8s;
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int row = 4 * (l >> 4) + i;
                        if (row < nrows) zdst[(size_t)prow[row] * P.zs + sig * a.r8max + j] = sc * acc[0][cb][i];
                    }
                }
            }
        }
        return;
    }

    // ---- base item: all rows x 64 columns over one K chunk
    b -= a.shrink_slots;
    int p = 0;
    while (p + 1 < a.n_proj && b >= a.p[p + 1].gemm_base) ++p;
    const DecProj& P = a.p[p];
    const int local = b - P.gemm_base;
    const int nt = local / P.ks, s = local - nt * P.ks;
    const int T = a.T, N = P.N;
    const int KS = P.K >> 5;
    const int nrb = (T + 15) >> 4, ncb = N >> 4;
    const uint16_t* ap[MB];
    const uint16_t* bp[2];
#pragma unroll
    for (int rb = 0; rb < MB; ++rb) ap[rb] = P.Xp + frag_index(min(rb, nrb - 1), 0, KS) + l * 8;
#pragma unroll
    for (int cb = 0; cb < 2; ++cb) bp[cb] = P.W + frag_index(min(nt * 4 + cg * 2 + cb, ncb - 1), 0, KS) + l * 8;
    f32x4 acc[MB][2];
    const int kb = s * P.kchunk;
    item_tile<MB>(acc, ap, bp, kb, min(KS, kb + P.kchunk), red);
    if (kq == 0) {
        float* ydst = P.Yp + (size_t)s * kDecodeMaxT * N;
#pragma unroll
        for (int cb = 0; cb < 2; ++cb) {
            const int col = nt * NT + cg * 32 + cb * 16 + lr;
            if (col < N) {
#pragma unroll
                for (int rb = 0; rb < MB; ++rb)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int row = rb * 16 + 4 * (l >> 4) + i;
                        if (row < T) ydst[(size_t)row * N + col] = acc[rb][cb][i];
                    }
            }
        }
    }
}

hipError_t launch_dec_main(const DecArgs& a, int mb, hipStream_t s) {
    const int grid = a.shrink_slots + a.gemm_items;
    if (grid <= 0) return hipSuccess;
    switch (mb) {
        case 1: hipLaunchKernelGGL(dec_main_kernel<1>, dim3(grid), dim3(kThreads), 0, s, a); break;
        case 2: hipLaunchKernelGGL(dec_main_kernel<2>, dim3(grid), dim3(kThreads), 0, s, a); break;
        case 3: hipLaunchKernelGGL(dec_main_kernel<3>, dim3(grid), dim3(kThreads), 0, s, a); break;
        case 4: hipLaunchKernelGGL(dec_main_kernel<4>, dim3(grid), dim3(kThreads), 0, s, a); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

__device__ __forceinline__ void add8(float (&acc)[8], const float* p) {
    const float4 a0 = *reinterpret_cast<const float4*>(p);
    const float4 a1 = *reinterpret_cast<const float4*>(p + 4);
    acc[0] += a0.x; acc[1] += a0.y; acc[2] += a0.z; acc[3] += a0.w;
    acc[4] += a1.x; acc[5] += a1.y; acc[6] += a1.z; acc[7] += a1.w;
}

// one thread = 8 consecutive outputs of one token row.  Every load of the
// thread is issued before the first use (split loops are unrolled to the
// largest split count and predicated).
__global__ __launch_bounds__(256) void dec_epi_kernel(DecArgs a) {
    const int u = blockIdx.x * 256 + threadIdx.x;
    if (u >= a.epi_units) return;
    int p = 0;
    while (p + 1 < a.n_proj && u >= a.p[p + 1].epi_base) ++p;
    const DecProj& P = a.p[p];
    const int per_row = P.N >> 3;
    const int local = u - P.epi_base;
    const int t = local / per_row, col = (local - t * per_row) * 8;
    const int ks = P.ks;
    const int v = a.vid[t];
    const int r8s = a.tr8[t];

    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    const float* y = P.Yp + (size_t)t * P.N + col;
#pragma unroll
    for (int s = 0; s < kMaxKSplit; ++s)
        if (s < ks) add8(acc, y + (size_t)s * kDecodeMaxT * P.N);

    if (r8s > 0) {
        int sig = 0;
        while (sig + 1 < P.n_slices && col >= P.slice_col[sig + 1]) ++sig;
        const float* z = P.Zp + (size_t)t * P.zs + sig * a.r8max;
        const uint16_t* bb = a.pool + (size_t)v * a.slot_stride + P.b_off + (size_t)col * r8s;
        // two 8-rank chunks per iteration, all their loads issued together
        for (int j0 = 0; j0 < r8s; j0 += 16) {
            const bool two = j0 + 8 < r8s;
            u32x4 q[2][8];
            float zz[2][8];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int jj = two ? j0 + 8 * h : j0;
#pragma unroll
                for (int c = 0; c < 8; ++c) q[h][c] = ld16(bb + (size_t)c * r8s + jj);
#pragma unroll
                for (int e = 0; e < 8; ++e) zz[h][e] = 0.f;
#pragma unroll
                for (int s = 0; s < kMaxKSplit; ++s)
                    if (s < ks) add8(zz[h], z + (size_t)s * kDecodeMaxT * P.zs + jj);
            }
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                if (h == 1 && !two) break;
#pragma unroll
                for (int c = 0; c < 8; ++c) {
                    const uint32_t qq[4] = {q[h][c].x, q[h][c].y, q[h][c].z, q[h][c].w};
                    float sum = 0.f;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        sum = fmaf(zz[h][2 * e], __uint_as_float(qq[e] << 16), sum);
                        sum = fmaf(zz[h][2 * e + 1], __uint_as_float(qq[e] & 0xffff0000u), sum);
                    }
                    acc[c] += sum;
                }
            }
        }
    }
    u32x4 o;
    o.x = (uint32_t)f2bf(acc[0]) | ((uint32_t)f2bf(acc[1]) << 16);
    o.y = (uint32_t)f2bf(acc[2]) | ((uint32_t)f2bf(acc[3]) << 16);
    o.z = (uint32_t)f2bf(acc[4]) | ((uint32_t)f2bf(acc[5]) << 16);
    o.w = (uint32_t)f2bf(acc[6]) | ((uint32_t)f2bf(acc[7]) << 16);
    *reinterpret_cast<u32x4*>(P.out + (size_t)t * P.N + col) = o;
}

hipError_t launch_dec_epi(const DecArgs& a, hipStream_t s) {
    const int grid = (a.epi_units + 255) / 256;
    if (grid <= 0) return hipSuccess;
    hipLaunchKernelGGL(dec_epi_kernel, dim3(grid), dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace bdl
