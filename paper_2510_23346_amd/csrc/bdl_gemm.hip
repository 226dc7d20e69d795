// Large-tile base GEMM with the fused BD-LoRA expand, for prefill batches.
//
// One workgroup computes a 256 x 256 output tile (tokens x columns) of one
// projection: out = X W_s + Zhat B, the base product, the adapter expand and
// their sum of Alg. 1 / Alg. 2 in one pass over the tile.  The operands are
// the packed fragment layouts (1 KB per 16 rows x 32 k), so a k-step of the
// tile is 16 activation and 16 weight fragments.  They go from global memory
// straight into LDS (buffer_load_dwordx4 ... lds: lane l of a wave writes the
// 16 bytes at offset 16 l of the wave's 1 KB destination, which is exactly a
// fragment), kBigStages k-steps deep, with one barrier per k-step.  Eight
// waves, 4 row quarters x 2 column halves, each own a 64 x 128 sub-tile for
// the whole K (no cross-wave reduction): per k-step a wave reads 4 + 8
// fragments from LDS (half a k-step ahead of the MFMAs that use them) and
// issues 32 MFMAs.  The MFMAs take the weight fragment as the A operand, so a
// lane ends up holding 4 consecutive output columns of one token and stores
// them with one 8-byte (bf16) or 16-byte (fp32) write.  The expand runs as
// extra MFMA k-steps over the 8-rank octets of the adapters present in the
// wave's 64 rows: each 16-lane group takes one octet (its own adapter, rows
// of other adapters masked to zero), the A operand is a slice of B^T_cat, the
// B operand the matching slice of scale * X A (a hi/lo bf16 pair, so the
// expand sees Z to about 16 bits).
//
// Rows: a tile's rows are positions in the plan's row order (tokens grouped
// by adapter, then the tokens without one), so a 64-row block carries few
// adapters; each lane gathers its activation row through its buffer-load
// offset, and Z and the output are addressed by token.
//
// Split tiles: when a batch has too few tiles for the chip, the host cuts a
// projection's tiles into ksplit k-ranges.  Each range stores its fp32 sum as
// a partial; a second launch of this kernel (fixup) adds a tile's partials
// in range order, then runs the expand and the store.
//
// Tile order: projections heaviest first (set by the host), inside a
// projection bands of kBigBand row tiles walked column by column.
#include "bdl_device.h"

namespace bdl {

constexpr int kBigFrags = 32;                    // fragments per k-step: 16 X + 16 W
constexpr int kBigStages = 4;                    // k-steps in LDS (32 KB each)
constexpr int kBigBand = 4;                      // row tiles per band of the tile order

typedef __attribute__((address_space(3))) void lds_void;

// Where this thread's copies of a k-step come from: copies i < CP / 2 are
// activation fragments, the others weight fragments (fragment w + NW i of
// the k-step's 32), each a buffer load of 16 bytes per lane at byte offset
// vo[i] + 1024 ks.  Buffer loads (not global ones) so that the compiler's
// wait-count bookkeeping treats them as plain vector-memory operations and
// keeps its LDS wait counts exact.
template <int CP>
struct BigSrc {
    __amdgpu_buffer_rsrc_t rx, rw;
    int vo[CP];   // this lane's byte offset at k-step 0
};

// issue this thread's CP fragment copies of k-step ks into one stage
template <int CP, int NW>
__device__ __forceinline__ void big_issue(const BigSrc<CP>& s, int ks, u32x4* stage, int w) {
#pragma unroll
    for (int i = 0; i < CP; ++i)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(i < CP / 2 ? s.rx : s.rw, (lds_void*)(stage + (w + NW * i) * 64), 16,
                                                 s.vo[i] + ks * 1024, 0, 0, 0);
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
    static_assert(n >= 0 && n < 64, "vmcnt field");
    __builtin_amdgcn_s_waitcnt((n & 15) | ((n >> 4) << 14) | (7 << 4));   // vmcnt(n) expcnt(7) lgkmcnt(0)
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(n) : "memory");
}

// wait until the k-step issued before the last `ahead` ones (0..3) is in LDS
template <int CP>
__device__ __forceinline__ void big_wait_ahead(int ahead) {
    if (ahead >= 3)
        big_wait_barrier<3 * CP>();
    else if (ahead == 2)
        big_wait_barrier<2 * CP>();
    else if (ahead == 1)
        big_wait_barrier<CP>();
    else
        big_wait_barrier<0>();
}

// RB = 16-row blocks per wave: 4 (eight waves, 4 x 2) or 8 (four waves, 2 x 2).
template <int RB>
__global__ __launch_bounds__(128 * (16 / RB)) void gemm_big_kernel(FwdArgs a) {
    constexpr int NWR = 16 / RB, NW = 2 * NWR;   // row waves, waves
    constexpr int CP = kBigFrags / NW;           // fragment copies per thread and k-step
    constexpr int NH = RB / 4;                   // 64-row blocks per wave
    __shared__ u32x4 lds[kBigStages * kBigFrags * 64];
    const int w = wave_id(), l = threadIdx.x & 63, lr = l & 15, lg = l >> 4;
    const int wr = w % NWR, wc = w / NWR;        // rows 16 RB wr .., columns 128 wc .. of the tile

    // Main launch: workgroup = one work item, a tile's k-range (split tiles
    // have ksplit items, item = tile * ksplit + range).  Fix-up launch:
    // workgroup = one split tile, whose partials it adds before the expand.
    const int bid = blockIdx.x;
    const bool fix = a.fixup != 0;
    if (bid >= (fix ? a.total_fix : a.total_tiles)) return;
    int p = 0;
#pragma unroll
    for (int q = 1; q < kMaxProjs; ++q)
        if (q < a.n_proj && (fix ? bid >= a.p[q].fix_base && a.p[q].fix_count > 0 : bid >= a.p[q].tile_base)) p = q;
    const ProjLaunch& P = a.p[p];
    const int S = P.ksplit;
    const int item = fix ? bid - P.fix_base : bid - P.tile_base;
    const int local = fix ? item : item / S, split = fix ? 0 : item - local * S;
    const int band = local / (kBigBand * P.tiles_n), off = local - band * kBigBand * P.tiles_n;
    const int bh = min(kBigBand, a.tiles_m - band * kBigBand);
    const int nt = off / bh, mt = band * kBigBand + (off - nt * bh);
    const int T = a.T, N = P.N, KS = P.K >> 5;
    const int nrb = (T + 15) >> 4, ncb = N >> 4;
    const int rbase = mt * kBigM + wr * 16 * RB; // first row of this wave
    const int c0 = nt * kBigN + wc * 128;        // first column of this wave

    // expand inputs that do not depend on the base product: fetched first.
    // Octet lists are per 64-row block; a block wholly past T has none.
    // Tile rows are positions in rowtok order (tokens grouped by adapter, so
    // a 64-row block holds few adapters and the expand few octets); tok[rb]
    // is the token of this lane's row of block rb (-1 past T).
    int code[NH], rvid[RB], tok[RB];
#pragma unroll
    for (int h = 0; h < NH; ++h) {
        const int* codes = a.tile_oct + (size_t)(mt * 4 + wr * NH + h) * a.oct_cap;
        code[h] = rbase + 64 * h < T ? codes[lg] : -1;
    }
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        const int row = rbase + rb * 16 + lr;
        // (clamped: a bad entry can cost a wrong row, never an access past X or out)
        tok[rb] = row < T ? (a.rowtok ? (int)min((unsigned)a.rowtok[row], (unsigned)(T - 1)) : row) : -1;
        rvid[rb] = tok[rb] >= 0 ? a.vid[tok[rb]] : -1;
    }

    f32x4 acc[RB][8];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int cb = 0; cb < 8; ++cb) acc[rb][cb] = f32x4{0.f, 0.f, 0.f, 0.f};
    // a split tile's partials: fp32, 16 bytes per lane per (wave, rb, cb),
    // kBigPartElems floats per partial, ksplit consecutive partials per tile
    const size_t part_lane = ((size_t)w * RB * 8) * 64 + l;
    f32x4* const part = reinterpret_cast<f32x4*>(a.bigpart) + (size_t)(P.part_base + local * S) * (kBigPartElems / 4);

    if (fix) {
        // partials in range order (fixed order: reproducible sums)
        for (int j = 0; j < S; ++j) {
            const f32x4* src = part + (size_t)j * (kBigPartElems / 4) + part_lane;
#pragma unroll
            for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                for (int cb = 0; cb < 8; ++cb) acc[rb][cb] += src[(rb * 8 + cb) * 64];
        }
    } else {
    // this item's k-steps [k0, k0 + NK)
    const int k0 = split * KS / S, NK = (split + 1) * KS / S - k0;

    // staging: fragments 0..15 of a k-step are the tile's activation row
    // blocks, 16..31 its weight column blocks (blocks past the edge are
    // clamped, their results are never stored)
    BigSrc<CP> src;
    src.rx = __builtin_amdgcn_make_buffer_rsrc((void*)P.Xp, 0, nrb * KS * 1024, kRawBufferWord3);
    src.rw = __builtin_amdgcn_make_buffer_rsrc((void*)P.W, 0, ncb * KS * 1024, kRawBufferWord3);
#pragma unroll
    for (int i = 0; i < CP; ++i) {
        const int f = w + NW * i;
        if (i < CP / 2 && a.rowtok) {
            // the lane's row is gathered: its token's fragment, lane slot
            // (token mod 16) + 16 (l / 16); rows past T repeat a valid token
            const int t = (int)min((unsigned)a.rowtok[min((mt * 16 + f) * 16 + lr, T - 1)], (unsigned)(T - 1));
            src.vo[i] = ((t >> 4) * KS + k0) * 1024 + ((t & 15) + 16 * lg) * 16;
        } else {
            src.vo[i] = (i < CP / 2 ? min(mt * 16 + f, nrb - 1) : min(nt * 16 + f - 16, ncb - 1)) * KS * 1024 +
                        k0 * 1024 + l * 16;
        }
    }
#pragma unroll
    for (int d = 0; d < kBigStages - 1; ++d)
        if (d < NK) big_issue<CP, NW>(src, d, lds + d * kBigFrags * 64, w);

    // Software pipeline over half k-steps (column blocks 0..3, then 4..7 of
    // the wave).  While the MFMAs of the first half run, the second half's
    // weight fragments are read from LDS; while those of the second half
    // run, the activation fragments and the first-half weight fragments of
    // the next k-step.  The barrier between the halves makes the next k-step
    // visible; the copies issued right after it refill the stage of k-step
    // ks - 1, whose LDS reads every wave finished before the previous barrier.
    static_assert(kBigStages >= 3 && kBigStages <= 5, "big_wait_ahead covers up to three k-steps in flight");
    auto stage = [&](int step) __attribute__((always_inline)) {
        return lds + (step % kBigStages) * kBigFrags * 64;
    };
    auto read_x = [&](u32x4 (&x)[RB], int step) __attribute__((always_inline)) {
        const u32x4* S0 = stage(step);
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) x[rb] = S0[(wr * RB + rb) * 64 + l];
    };
    auto read_w = [&](u32x4 (&wv)[4], int step, int half) __attribute__((always_inline)) {
        const u32x4* S0 = stage(step);
#pragma unroll
        for (int c = 0; c < 4; ++c) wv[c] = S0[(16 + wc * 8 + 4 * half + c) * 64 + l];
    };
    auto mma = [&](const u32x4 (&x)[RB], const u32x4 (&wv)[4], int half) __attribute__((always_inline)) {
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
            for (int c = 0; c < 4; ++c)
                acc[rb][4 * half + c] = mfma(wv[c], x[rb], acc[rb][4 * half + c]);
    };
    u32x4 xa[RB], xb[RB], w0[4], w1[4];
    // k-step ks < NK - 1 (x holds its activations, w0 its first-half
    // weights; the next k-step's activations arrive in xn)
    // (the scheduling groups pin the reads ahead of the MFMAs they overlap:
    // masks 0x100 = LDS read, 0x008 = MFMA)
    auto k_step = [&](int ks, const u32x4 (&x)[RB], u32x4 (&xn)[RB]) __attribute__((always_inline)) {
        read_w(w1, ks, 1);
        mma(x, w0, 0);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, 4 * RB - 4, 0);
        __builtin_amdgcn_sched_barrier(0);
        // k-step ks + 1 is complete once at most the copies issued after it
        // (k-steps ks + 2 .. ks + kBigStages - 2 below NK) are in flight
        big_wait_ahead<CP>(min(kBigStages - 3, NK - 2 - ks));
        const int nx = ks + kBigStages - 1;
        if (nx < NK) big_issue<CP, NW>(src, nx, stage(nx), w);
        read_x(xn, ks + 1);
        read_w(w0, ks + 1, 0);
        mma(x, w1, 1);
        // RB + 4 reads spread over the 4 RB MFMAs
#pragma unroll
        for (int i = 0; i < RB + 4; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, (4 * RB) / (RB + 4) > 0 ? (4 * RB) / (RB + 4) : 1, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
    };
    // k-step 0 is complete once at most the copies of k-steps 1 .. kBigStages - 2 are in flight
    big_wait_ahead<CP>(min(kBigStages - 2, NK - 1));
    read_x(xa, 0);
    read_w(w0, 0, 0);
    int ks = 0;
    for (; ks + 2 < NK; ks += 2) {
        k_step(ks, xa, xb);
        k_step(ks + 1, xb, xa);
    }
    // one or two k-steps left; the last one reads nothing ahead
    const bool two = ks + 1 < NK;
    if (two) k_step(ks, xa, xb);
    const u32x4 (&xl)[RB] = two ? xb : xa;
    read_w(w1, NK - 1, 1);
    mma(xl, w0, 0);
    mma(xl, w1, 1);
    if (S > 1) {
        // a range of a split tile: store the partial, the fix-up launch adds it
        f32x4* dst = part + (size_t)split * (kBigPartElems / 4) + part_lane;
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
            for (int cb = 0; cb < 8; ++cb) dst[(rb * 8 + cb) * 64] = acc[rb][cb];
        return;
    }
    }

    // expand: acc += Zhat B over the octets of each 64-row block of the wave
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
#pragma unroll
    for (int h = 0; h < NH; ++h) {
        const int* codes = a.tile_oct + (size_t)(mt * 4 + wr * NH + h) * a.oct_cap;
        int cd = code[h];
        for (int e = 0;;) {
            if (!__any(cd >= 0)) break;
            const int slot = cd >> 12, r8s = (cd >> 4) & 0xff, j0 = (cd & 15) * 8;
            u32x4 bv[8];
#pragma unroll
            for (int cb = 0; cb < 8; ++cb) {
                const int col = min(c0 + cb * 16 + lr, N - 1);
                bv[cb] = cd >= 0 ? ld16(a.pool + (size_t)slot * a.slot_stride + P.b_off + (size_t)col * r8s + j0)
                                 : zero4;
            }
            u32x4 zh[4], zl[4];
#pragma unroll
            for (int cb = 0; cb < 8; ++cb) {
                if (cb == 0 || sig[cb] != sig[cb - 1]) {
#pragma unroll
                    for (int rb = 0; rb < 4; ++rb) {
                        const bool match = cd >= 0 && rvid[4 * h + rb] == slot;
                        const uint16_t* zp =
                            P.Z + (size_t)max(tok[4 * h + rb], 0) * P.zs + sig[cb] * a.r8max + j0;
                        zh[rb] = match ? ld16(zp) : zero4;
                        zl[rb] = match ? ld16(zp + P.zplane) : zero4;
                    }
                }
#pragma unroll
                for (int rb = 0; rb < 4; ++rb) {
                    acc[4 * h + rb][cb] = mfma(bv[cb], zh[rb], acc[4 * h + rb][cb]);
                    acc[4 * h + rb][cb] = mfma(bv[cb], zl[rb], acc[4 * h + rb][cb]);
                }
            }
            e += 4;
            if (e + 4 > a.oct_cap) break;
            cd = codes[e + lg];
        }
    }

    // store: lane (lr, lg) of block (rb, cb) holds row rbase + 16 rb + lr
    // (token tok[rb]), columns c0 + 16 cb + 4 lg + i
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        const int row = tok[rb];
        if (row < 0) continue;
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

// wave tile height of the launch: 4 row blocks (eight waves of 64 x 128)
constexpr int kBigRB = 4;

hipError_t launch_gemm_big(const FwdArgs& a, hipStream_t s) {
    if (a.total_tiles <= 0) return hipSuccess;
    hipLaunchKernelGGL(gemm_big_kernel<kBigRB>, dim3(a.total_tiles), dim3(128 * (16 / kBigRB)), 0, s, a);
    if (a.total_fix > 0) {
        FwdArgs f = a;
        f.fixup = 1;
        hipLaunchKernelGGL(gemm_big_kernel<kBigRB>, dim3(a.total_fix), dim3(128 * (16 / kBigRB)), 0, s, f);
    }
    return hipGetLastError();
}

}  // namespace bdl
