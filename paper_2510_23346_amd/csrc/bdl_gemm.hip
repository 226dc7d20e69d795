// Large-tile base GEMM with the fused BD-LoRA expand, for prefill batches.
//
// One workgroup computes a 256 x 256 output tile (tokens x columns) of one
// projection: out = X W_s + Zhat B, the base product, the adapter expand and
// their sum of Alg. 1 / Alg. 2 in one pass over the tile.  The operands are
// the packed fragment layouts (1 KB per 16 rows x 32 k), so a k-step of the
// tile is 16 activation and 16 weight fragments.  They go from global memory
// straight into LDS (global_load_lds_dwordx4: lane l of a wave writes the
// 16 bytes at offset 16 l of the wave's 1 KB destination, which is exactly a
// fragment), kBigStages k-steps deep, with one barrier per k-step.  Eight
// waves, 4 row quarters x 2 column halves, each own a 64 x 128 sub-tile for
// the whole K (no cross-wave reduction): per k-step a wave reads 4 + 8
// fragments from LDS (one k-step ahead, into a second register set) and
// issues 32 MFMAs.  The MFMAs take the weight fragment as the A operand, so a
// lane ends up holding 4 consecutive output columns of one token and stores
// them with one 8-byte (bf16) or 16-byte (fp32) write.  The expand runs as
// extra MFMA k-steps over the 8-rank octets of the adapters present in the
// wave's 64 rows: each 16-lane group takes one octet (its own adapter, rows
// of other adapters masked to zero), the A operand is a slice of B^T_cat, the
// B operand the matching slice of scale * X A (a hi/lo bf16 pair, so the
// expand sees Z to about 16 bits).
//
// Tile order: projections heaviest first (set by the host), inside a
// projection bands of kBigBand row tiles walked column by column, so that
// the workgroups running at one time share activation rows and weight
// columns.
#include "bdl_device.h"

namespace bdl {

constexpr int kBigThreads = 512;
constexpr int kBigFrags = 32;                    // fragments per k-step: 16 X + 16 W
constexpr int kBigStages = 4;                    // k-steps in LDS (32 KB each)
constexpr int kBigBand = 4;                      // row tiles per band of the tile order

typedef __attribute__((address_space(3))) void lds_void;

// the LDS fragments one wave multiplies in one k-step
struct BigFrags {
    u32x4 x[4];   // activation row blocks 4 wr .. 4 wr + 3
    u32x4 w[8];   // weight column blocks 8 wc .. 8 wc + 7
};

// issue the 4 fragment copies of this thread for one k-step into one stage
__device__ __forceinline__ void big_issue(const uint16_t* const (&src)[4], size_t koff, u32x4* stage, int w) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
        __builtin_amdgcn_global_load_lds(static_cast<const void*>(src[i] + koff),
                                         (lds_void*)(stage + (w + 8 * i) * 64), 16, 0, 0);
}

// wait until at most n of this thread's copies (and none of its LDS reads)
// are in flight, then barrier: afterwards the k-step whose copies are older
// than those n is in LDS for every wave, and every wave has finished reading
// the fragments it loaded before.  The builtin wait tells the compiler's own
// counter tracking what has completed; the barrier is inline assembly with a
// memory clobber so that no LDS access moves across it (the wait is repeated
// there, which costs nothing once satisfied).
template <int n>
__device__ __forceinline__ void big_wait_barrier() {
    static_assert(n >= 0 && n < 16, "vmcnt field");
    __builtin_amdgcn_s_waitcnt(n | (7 << 4));   // vmcnt(n) expcnt(7) lgkmcnt(0)
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(n) : "memory");
}

__global__ __launch_bounds__(kBigThreads) void gemm_big_kernel(FwdArgs a) {
    __shared__ u32x4 lds[kBigStages * kBigFrags * 64];
    const int w = wave_id(), l = threadIdx.x & 63, lr = l & 15, lg = l >> 4;
    const int wr = w & 3, wc = w >> 2;           // rows 64 wr .., columns 128 wc .. of the tile

    const int bid = blockIdx.x;
    int p = 0;
#pragma unroll
    for (int q = 1; q < kMaxProjs; ++q)
        if (q < a.n_proj && bid >= a.p[q].tile_base) p = q;
    const ProjLaunch& P = a.p[p];
    const int local = bid - P.tile_base;
    const int band = local / (kBigBand * P.tiles_n), off = local - band * kBigBand * P.tiles_n;
    const int bh = min(kBigBand, a.tiles_m - band * kBigBand);
    const int nt = off / bh, mt = band * kBigBand + (off - nt * bh);
    const int T = a.T, N = P.N, KS = P.K >> 5;
    const int nrb = (T + 15) >> 4, ncb = N >> 4;
    const int rbase = mt * kBigM + wr * 64;      // first row of this wave
    const int c0 = nt * kBigN + wc * 128;        // first column of this wave

    // expand inputs that do not depend on the base product: fetched first.
    // Octet lists are per 64-row block; a wave wholly past T has none.
    const int* codes = a.tile_oct + (size_t)(mt * 4 + wr) * a.oct_cap;
    int code = rbase < T ? codes[lg] : -1;
    int rvid[4];
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
        const int row = rbase + rb * 16 + lr;
        rvid[rb] = row < T ? a.vid[row] : -1;
    }

    // staging: this thread copies lane l of fragments w + 8 i (i = 0..3) of
    // every k-step; fragments 0..15 are the tile's activation row blocks,
    // 16..31 its weight column blocks (blocks past the edge are clamped, their
    // results are never stored)
    const uint16_t* src[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int f = w + 8 * i;
        src[i] = (f < 16 ? P.Xp + frag_index(min(mt * 16 + f, nrb - 1), 0, KS)
                         : P.W + frag_index(min(nt * 16 + f - 16, ncb - 1), 0, KS)) + l * 8;
    }
#pragma unroll
    for (int d = 0; d < kBigStages - 1; ++d)
        if (d < KS) big_issue(src, (size_t)d * kFrag, lds + d * kBigFrags * 64, w);

    f32x4 acc[4][8];
#pragma unroll
    for (int rb = 0; rb < 4; ++rb)
#pragma unroll
        for (int cb = 0; cb < 8; ++cb) acc[rb][cb] = f32x4{0.f, 0.f, 0.f, 0.f};

    // Software pipeline over half k-steps (column blocks 0..3, then 4..7 of
    // the wave).  While the MFMAs of the first half run, the second half's
    // weight fragments are read from LDS; while those of the second half
    // run, the activation fragments and the first-half weight fragments of
    // the next k-step.  The barrier between the halves makes the next k-step
    // visible; the copies issued right after it refill the stage of k-step
    // ks - 1, whose LDS reads every wave finished before the previous barrier.
    static_assert(kBigStages == 4, "the waits below are written for four stages");
    auto stage = [&](int step) __attribute__((always_inline)) {
        return lds + (step % kBigStages) * kBigFrags * 64;
    };
    auto read_x = [&](u32x4 (&x)[4], int step) __attribute__((always_inline)) {
        const u32x4* S0 = stage(step);
#pragma unroll
        for (int rb = 0; rb < 4; ++rb) x[rb] = S0[(wr * 4 + rb) * 64 + l];
    };
    auto read_w = [&](u32x4 (&wv)[4], int step, int half) __attribute__((always_inline)) {
        const u32x4* S0 = stage(step);
#pragma unroll
        for (int c = 0; c < 4; ++c) wv[c] = S0[(16 + wc * 8 + 4 * half + c) * 64 + l];
    };
    auto mma = [&](const u32x4 (&x)[4], const u32x4 (&wv)[4], int half) __attribute__((always_inline)) {
#pragma unroll
        for (int rb = 0; rb < 4; ++rb)
#pragma unroll
            for (int c = 0; c < 4; ++c)
                acc[rb][4 * half + c] = mfma(wv[c], x[rb], acc[rb][4 * half + c]);
    };
    u32x4 xa[4], xb[4], w0[4], w1[4];
    // k-step ks < KS - 1 (x holds its activations, w0 its first-half weights)
    // (the scheduling groups pin the reads ahead of the MFMAs they overlap:
    // masks 0x100 = LDS read, 0x008 = MFMA)
    auto k_step = [&](int ks, const u32x4 (&x)[4], u32x4 (&xn)[4]) __attribute__((always_inline)) {
        read_w(w1, ks, 1);
        mma(x, w0, 0);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, 12, 0);
        __builtin_amdgcn_sched_barrier(0);
        // k-step ks + 1 is complete once at most the copies of ks + 2 are in flight
        if (ks + 2 < KS)
            big_wait_barrier<4>();
        else
            big_wait_barrier<0>();
        const int nx = ks + kBigStages - 1;
        if (nx < KS) big_issue(src, (size_t)nx * kFrag, stage(nx), w);
        read_x(xn, ks + 1);
        read_w(w0, ks + 1, 0);
        mma(x, w1, 1);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
    };
    // k-step 0 is complete once at most the copies of k-steps 1 and 2 are in flight
    if (KS >= 3)
        big_wait_barrier<8>();
    else if (KS == 2)
        big_wait_barrier<4>();
    else
        big_wait_barrier<0>();
    read_x(xa, 0);
    read_w(w0, 0, 0);
    int ks = 0;
    for (; ks + 2 < KS; ks += 2) {
        k_step(ks, xa, xb);
        k_step(ks + 1, xb, xa);
    }
    // one or two k-steps left; the last one reads nothing ahead
    const bool two = ks + 1 < KS;
    if (two) k_step(ks, xa, xb);
    const u32x4 (&xl)[4] = two ? xb : xa;
    read_w(w1, KS - 1, 1);
    mma(xl, w0, 0);
    mma(xl, w1, 1);

    // expand: acc += Zhat B over the octets of this wave's 64 rows
    int sig[8];
#pragma unroll
    for (int cb = 0; cb < 8; ++cb) {
        const int c = c0 + cb * 16;
        int sgm = 0;
#pragma unroll
        for (int q = 1; q < kMaxSlices; ++q)
            if (q < P.n_slices && c >= P.slice_col[q]) sgm = q;
        sig[cb] = sgm;
    }
    const u32x4 zero4 = u32x4{0u, 0u, 0u, 0u};
    for (int e = 0;;) {
        if (!__any(code >= 0)) break;
        const int slot = code >> 12, r8s = (code >> 4) & 0xff, j0 = (code & 15) * 8;
        u32x4 bv[8];
#pragma unroll
        for (int cb = 0; cb < 8; ++cb) {
            const int col = min(c0 + cb * 16 + lr, N - 1);
            bv[cb] = code >= 0 ? ld16(a.pool + (size_t)slot * a.slot_stride + P.b_off + (size_t)col * r8s + j0)
                               : zero4;
        }
        u32x4 zh[4], zl[4];
#pragma unroll
        for (int cb = 0; cb < 8; ++cb) {
            if (cb == 0 || sig[cb] != sig[cb - 1]) {
#pragma unroll
                for (int rb = 0; rb < 4; ++rb) {
                    const bool match = code >= 0 && rvid[rb] == slot;
                    const uint16_t* zp = P.Z + (size_t)(rbase + rb * 16 + lr) * P.zs + sig[cb] * a.r8max + j0;
                    zh[rb] = match ? ld16(zp) : zero4;
                    zl[rb] = match ? ld16(zp + P.zplane) : zero4;
                }
            }
#pragma unroll
            for (int rb = 0; rb < 4; ++rb) {
                acc[rb][cb] = mfma(bv[cb], zh[rb], acc[rb][cb]);
                acc[rb][cb] = mfma(bv[cb], zl[rb], acc[rb][cb]);
            }
        }
        e += 4;
        if (e + 4 > a.oct_cap) break;
        code = codes[e + lg];
    }

    // store: lane (lr, lg) of block (rb, cb) holds row rbase + 16 rb + lr,
    // columns c0 + 16 cb + 4 lg + i
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
        const int row = rbase + rb * 16 + lr;
        if (row >= T) continue;
#pragma unroll
        for (int cb = 0; cb < 8; ++cb) {
            const int col = c0 + cb * 16 + 4 * lg;
            if (col >= N) continue;
            const f32x4 v = acc[rb][cb];
            if (P.out_f32) {
                *reinterpret_cast<f32x4*>(P.out_f32 + (size_t)row * N + col) = v;
            } else {
                const uint32_t lo = (uint32_t)f2bf(v[0]) | ((uint32_t)f2bf(v[1]) << 16);
                const uint32_t hi = (uint32_t)f2bf(v[2]) | ((uint32_t)f2bf(v[3]) << 16);
                *reinterpret_cast<uint2*>(P.out + (size_t)row * N + col) = make_uint2(lo, hi);
            }
        }
    }
}

hipError_t launch_gemm_big(const FwdArgs& a, hipStream_t s) {
    if (a.total_tiles <= 0) return hipSuccess;
    hipLaunchKernelGGL(gemm_big_kernel, dim3(a.total_tiles), dim3(kBigThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace bdl
