// Base GEMMs of batches above the decode size, bf16 weights: the large-tile
// GEMM with the fused BD-LoRA expand (prefill batches, below), and the
// medium-batch GEMM with its epilogue (further down).
//
// Large-tile GEMM.
// One workgroup computes a 256 x 256 output tile (tokens x columns) of one
// projection: out = X W_s + Zhat B, the base product, the adapter expand and
// their sum of Alg. 1 / Alg. 2 in one pass over the tile.  A k-step of the
// tile is 16 activation and 16 weight fragments (1 KB per 16 rows x 32 k).
// They go from global memory straight into LDS (buffer_load_dwordx4 ... lds:
// lane l of a wave writes the 16 bytes at offset 16 l of the wave's 1 KB
// destination), with one barrier per k-step.  The weight is read in its
// packed fragment layout, a k-step per slot of a ring of kBigStages slots.
// The activations come straight from the caller's row-major X (no pass packs
// X first): a copy takes 8 rows x 128 bytes, the two k-steps of a pair, each
// lane's global offset picking 16 bytes of its token's row, into a ring of
// pair slots beside the weights' ring; or, when X is an intermediate already
// written in fragments, from that packed copy, a k-step per stage of one
// ring.  A k-step's refills are issued after its MFMAs.  Eight
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

// Where this thread's copies come from: copies i < CP / 2 of a k-step are
// activation fragments, the others weight fragments (fragment w + NW i of
// the k-step's 32), each a buffer load of 16 bytes per lane at byte offset
// vo[i] + 1024 ks (weights, packed X); with row-major X the activation
// copies of pair q are at xo[j] + 128 q instead (see big_issue_x).  Buffer
// loads (not global ones) so that the
// compiler's wait-count bookkeeping treats them as plain vector-memory
// operations and keeps its LDS wait counts exact; their bounds are the
// operands' sizes, so no lane can read past X or W.
template <int CP>
struct BigSrc {
    __amdgpu_buffer_rsrc_t rx, rw, rw2;
    int vo[CP];   // this lane's byte offset at k-step 0
    int xo[CP];   // row-major X: this lane's offsets of its CP half-fragment copies of pair 0
    bool two[CP]; // paired gate/up tiles: the copy reads the second weight (rw2)
};

// issue this thread's CP fragment copies of k-step ks into one stage
template <int CP, int NW>
__device__ __forceinline__ void big_issue(const BigSrc<CP>& s, int ks, u32x4* stage, int w) {
#pragma unroll
    for (int i = 0; i < CP; ++i)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(i < CP / 2 ? s.rx : (s.two[i] ? s.rw2 : s.rw),
                                                 (lds_void*)(stage + (w + NW * i) * 64), 16, s.vo[i] + ks * 1024, 0,
                                                 0, 0);
}

// Row-major X (the caller's activations): one copy takes 8 rows x 128 bytes
// of the tile, the two k-steps of a pair (whole lines).  A pair's 32 copies
// (16 row blocks x 2 row halves) land in one slot of an activation ring, half
// fragment h = 2 block + half at 1 KB each; lane l takes row l / 8 of its 8
// and 16-byte chunk (l mod 8) ^ big_swz(row of the block), so that the
// readers hit distinct LDS banks (16 lanes on distinct 16-byte bank groups
// mod 16, each 8 of them mod 8).  The weights keep one k-step per slot of
// their own ring.
__device__ __forceinline__ int big_swz(int r) { return ((r >> 1) ^ ((r & 1) << 2)) & 7; }

// the weight copies (i >= CP / 2) of k-step ks into its weight slot (16 fragments)
template <int CP, int NW>
__device__ __forceinline__ void big_issue_w(const BigSrc<CP>& s, int ks, u32x4* slot, int w) {
#pragma unroll
    for (int i = CP / 2; i < CP; ++i)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(s.two[i] ? s.rw2 : s.rw, (lds_void*)(slot + (w + NW * i - 16) * 64),
                                                 16, s.vo[i] + ks * 1024, 0, 0, 0);
}

// this thread's CP copies of activation pair q into its slot (32 half fragments)
template <int CP, int NW>
__device__ __forceinline__ void big_issue_x(const BigSrc<CP>& s, int q, u32x4* slot, int w) {
#pragma unroll
    for (int j = 0; j < CP; ++j)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(s.rx, (lds_void*)(slot + (w + NW * j) * 64), 16, s.xo[j] + q * 128, 0,
                                                 0, 0);
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

// wait until at most n (0, 2, 4 or 6) of this thread's copies are in flight, then barrier
__device__ __forceinline__ void big_wait_n(int n) {
    if (n >= 6)
        big_wait_barrier<6>();
    else if (n >= 4)
        big_wait_barrier<4>();
    else if (n >= 2)
        big_wait_barrier<2>();
    else
        big_wait_barrier<0>();
}

// RB = 16-row blocks per wave: 4 (eight waves, 4 x 2) or 8 (four waves, 2 x 2).
// XRM: the activations come from the caller's row-major X in pairs of
// k-steps (see big_issue_x), in a ring of kBigXPairs pair slots beside the
// weights' ring of kBigStages k-step slots (all of the CU's 160 KB of LDS);
// a pair is copied 4 k-steps ahead of its first k-step, so it is in LDS
// before the weights of that k-step are.
constexpr int kBigXPairs = 3;
template <int RB, bool XRM>
__global__ __launch_bounds__(128 * (16 / RB)) void gemm_big_kernel(FwdArgs a) {
    constexpr int NWR = 16 / RB, NW = 2 * NWR;   // row waves, waves
    constexpr int CP = kBigFrags / NW;           // fragment copies per thread and k-step
    constexpr int NH = RB / 4;                   // 64-row blocks per wave
    constexpr int ST = kBigStages;               // k-step stages (weight slots)
    static_assert(!XRM || (NW == 8 && CP == 4), "the row-major form's wait counts assume 8 waves");
    __shared__ u32x4 lds[(XRM ? ST * 16 + kBigXPairs * 32 : ST * kBigFrags) * 64];
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
    // Paired tiles (the MLP's gate and up, equal shapes): the tile's 256
    // columns are gate columns nt 128 .. + 127 (waves of column half 0) and
    // the same up columns (half 1), so that H = silu(gate) * up is formed in
    // the workgroup.  Projection p is gate, p + 1 up.
    const bool pair = a.mlp_act == BDLORA_ACT_SILU_MUL;
    const int c0 = pair ? nt * 128 : nt * kBigN + wc * 128;   // first column of this wave
    const ProjLaunch& Pe = a.p[p + (pair && wc == 1 ? 1 : 0)];  // this wave's projection

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
    // this item's k-steps [k0, k0 + NK); row-major X: even bounds, so every
    // pair of k-steps starts a 128-byte line (the host keeps KS even and
    // each range at least 2 k-steps long)
    int k0 = split * KS / S, k1 = (split + 1) * KS / S;
    if (XRM) {
        k0 &= ~1;
        k1 = split + 1 == S ? KS : k1 & ~1;
    }
    const int NK = k1 - k0;

    // staging: fragments 0..15 of a k-step are the tile's activation row
    // blocks, 16..31 its weight column blocks (blocks past the edge are
    // clamped, their results are never stored)
    BigSrc<CP> src;
    src.rx = XRM ? __builtin_amdgcn_make_buffer_rsrc((void*)P.X, 0, T * P.K * 2, kRawBufferWord3)
                 : __builtin_amdgcn_make_buffer_rsrc((void*)P.Xp, 0, nrb * KS * 1024, kRawBufferWord3);
    src.rw = __builtin_amdgcn_make_buffer_rsrc((void*)P.W, 0, ncb * KS * 1024, kRawBufferWord3);
    src.rw2 = pair ? __builtin_amdgcn_make_buffer_rsrc((void*)a.p[p + 1].W, 0, ncb * KS * 1024, kRawBufferWord3)
                   : src.rw;
#pragma unroll
    for (int i = 0; i < CP; ++i) {
        const int f = w + NW * i;
        src.two[i] = pair && i >= CP / 2 && f - 16 >= 8;
        src.xo[i] = 0;
        if (i >= CP / 2 && pair) {
            // weight fragment f - 16: column block (f - 16) mod 8 of gate (< 8) or up
            src.vo[i] = min(nt * 8 + ((f - 16) & 7), ncb - 1) * KS * 1024 + k0 * 1024 + l * 16;
        } else if (i < CP / 2 && XRM) {
            // (row-major X: src.xo below)
        } else if (i < CP / 2 && a.rowtok) {
            // the lane's row is gathered: its token's fragment, lane slot
            // (token mod 16) + 16 (l / 16); rows past T repeat a valid token
            const int t = (int)min((unsigned)a.rowtok[min((mt * 16 + f) * 16 + lr, T - 1)], (unsigned)(T - 1));
            src.vo[i] = ((t >> 4) * KS + k0) * 1024 + ((t & 15) + 16 * lg) * 16;
        } else {
            src.vo[i] = (i < CP / 2 ? min(mt * 16 + f, nrb - 1) : min(nt * 16 + f - 16, ncb - 1)) * KS * 1024 +
                        k0 * 1024 + l * 16;
        }
    }
    if constexpr (XRM) {
        // half fragment h = w + NW j of a pair: row block h / 2, rows 8 (h mod 2)
        // + l / 8 (its token; rows past T repeat a valid one), chunk
        // (l mod 8) ^ big_swz(row in block) of the pair's 128 bytes from input 32 k0
#pragma unroll
        for (int j = 0; j < CP; ++j) {
            const int h = w + NW * j, rr = 8 * (h & 1) + (l >> 3);
            const int row = min((mt * 16 + (h >> 1)) * 16 + rr, T - 1);
            const int t = a.rowtok ? (int)min((unsigned)a.rowtok[row], (unsigned)(T - 1)) : row;
            src.xo[j] = t * (P.K * 2) + k0 * 64 + ((l & 7) ^ big_swz(rr)) * 16;
        }
    }
    u32x4* const wring = lds;                     // row-major X: weight slots, then pair slots
    u32x4* const xring = lds + ST * 16 * 64;
    const int NP = NK >> 1;                       // row-major X: pairs (NK is even)
    if constexpr (XRM) {
        // pairs 0 and 1, then the weights of k-steps 0 .. ST - 2
#pragma unroll
        for (int q = 0; q < 2; ++q)
            if (q < NP) big_issue_x<CP, NW>(src, q, xring + q * 32 * 64, w);
#pragma unroll
        for (int d = 0; d < ST - 1; ++d)
            if (d < NK) big_issue_w<CP, NW>(src, d, wring + d * 16 * 64, w);
    } else {
#pragma unroll
        for (int d = 0; d < ST - 1; ++d)
            if (d < NK) big_issue<CP, NW>(src, d, lds + d * kBigFrags * 64, w);
    }

    // Software pipeline over half k-steps (column blocks 0..3, then 4..7 of
    // the wave).  While the MFMAs of the first half run, the second half's
    // weight fragments are read from LDS; while those of the second half
    // run, the activation fragments and the first-half weight fragments of
    // the next k-step.  The barrier between the halves makes the next k-step
    // visible; the copies issued right after it refill the stage of k-step
    // ks - 1, whose LDS reads every wave finished before the previous barrier.
    static_assert(ST >= 3 && ST <= 5, "big_wait_ahead covers up to three k-steps in flight");
    auto stage = [&](int step) __attribute__((always_inline)) {
        return lds + (step % ST) * kBigFrags * 64;
    };
    // row-major X: lane (lr, lg) of k-step 2 p + h finds its 8 inputs (row
    // lr, chunk 4 h + lg of the pair) in pair p's slot, half fragment
    // 2 block + lr / 8, position 8 (lr mod 8) + ((4 h + lg) ^ big_swz(lr))
    const int xpos0 = (lr >> 3) * 64 + (lr & 7) * 8 + (lg ^ big_swz(lr));
    const int xpos1 = (lr >> 3) * 64 + (lr & 7) * 8 + ((4 + lg) ^ big_swz(lr));
    auto read_x = [&](u32x4 (&x)[RB], int step) __attribute__((always_inline)) {
        if constexpr (XRM) {
            const u32x4* S0 = xring + ((step >> 1) % kBigXPairs) * 32 * 64 + ((step & 1) ? xpos1 : xpos0);
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) x[rb] = S0[(wr * RB + rb) * 128];
        } else {
            const u32x4* S0 = stage(step);
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) x[rb] = S0[(wr * RB + rb) * 64 + l];
        }
    };
    auto read_w = [&](u32x4 (&wv)[4], int step, int half) __attribute__((always_inline)) {
        if constexpr (XRM) {
            const u32x4* S0 = wring + (step % ST) * 16 * 64;
#pragma unroll
            for (int c = 0; c < 4; ++c) wv[c] = S0[(wc * 8 + 4 * half + c) * 64 + l];
        } else {
            const u32x4* S0 = stage(step);
#pragma unroll
            for (int c = 0; c < 4; ++c) wv[c] = S0[(16 + wc * 8 + 4 * half + c) * 64 + l];
        }
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
        const int nx = ks + ST - 1;
        if constexpr (XRM) {
            // k-step ks + 1's weights are complete once at most the copies
            // issued after them are in flight: the weights of ks + 2 (if any)
            // and, after an even k-step, the pair issued there; its pair was
            // issued before its weights
            big_wait_n((ks + 2 <= NK - 1 ? 2 : 0) + ((ks & 1) && ((ks - 1) >> 1) + 2 < NP ? 4 : 0));
        } else {
            // k-step ks + 1 is complete once at most the copies issued after it
            // (k-steps ks + 2 .. ks + ST - 2 below NK) are in flight
            big_wait_ahead<CP>(min(ST - 3, NK - 2 - ks));
            if (nx < NK) big_issue<CP, NW>(src, nx, stage(nx), w);
        }
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
        if constexpr (XRM) {
            // the refills of the slots freed at this k-step's barrier follow
            // its MFMAs: issued in a burst ahead of them they held them up
            // (the next barrier's waits count them the same either way)
            if (!(ks & 1) && (ks >> 1) + 2 < NP)
                big_issue_x<CP, NW>(src, (ks >> 1) + 2, xring + (((ks >> 1) + 2) % kBigXPairs) * 32 * 64, w);
            if (nx < NK) big_issue_w<CP, NW>(src, nx, wring + (nx % ST) * 16 * 64, w);
        }
    };
    // k-step 0 is complete once at most the copies of k-steps 1 .. ST - 2 are
    // in flight (row-major X: the weights of k-steps 1 .. ST - 2; the pairs
    // were issued first)
    if (XRM)
        big_wait_n(2 * min(ST - 2, NK - 1));
    else
        big_wait_ahead<CP>(min(ST - 2, NK - 1));
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
            if (q < Pe.n_slices && c >= Pe.slice_col[q]) sgm = q;
        sig[cb] = sgm;
    }
    const u32x4 zero4 = u32x4{0u, 0u, 0u, 0u};
#pragma unroll
    for (int h = 0; h < NH; ++h) {
        const int* codes = a.tile_oct + (size_t)(mt * 4 + wr * NH + h) * a.oct_cap;
        int cd = code[h];
        for (int e = 0;;) {
            if (!__any(cd >= 0)) break;
            // the next four codes, in flight with this turn's operands
            const int cdn = e + 8 <= a.oct_cap ? codes[e + 4 + lg] : -1;
            const int slot = cd >> 12, r8s = (cd >> 4) & 0xff, j0 = (cd & 15) * 8;
            u32x4 bv[8];
#pragma unroll
            for (int cb = 0; cb < 8; ++cb) {
                const int col = min(c0 + cb * 16 + lr, N - 1);
                bv[cb] = cd >= 0 ? ld16(a.pool + (size_t)slot * a.slot_stride + Pe.b_off + (size_t)col * r8s + j0)
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
                            Pe.Z + (size_t)max(tok[4 * h + rb], 0) * Pe.zs + sig[cb] * a.r8max + j0;
                        zh[rb] = match ? ld16(zp) : zero4;
                        zl[rb] = match ? ld16(zp + Pe.zplane) : zero4;
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
            cd = cdn;
        }
    }

    // store: lane (lr, lg) of block (rb, cb) holds row rbase + 16 rb + lr
    // (token tok[rb]), columns c0 + 16 cb + 4 lg + i
    if (a.mlp_act >= 0) {
        // the MLP intermediate: H in bf16, once, in the fragment layout of the
        // second projection's input (element [(t/16 KS + c/32) 512 + (t%16 +
        // 16 ((c%32)/8)) 8 + c%8] for token t, column c); the 4 columns of a
        // lane are contiguous there.  Paired tiles first hand the up values to
        // the gate waves through LDS (the k-loop's stages are free: every
        // copy has landed and every wave is past its last read).
        f32x4* xl = reinterpret_cast<f32x4*>(lds);
        if (pair) {
            __syncthreads();
            if (wc == 1) {
#pragma unroll
                for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                    for (int cb = 0; cb < 8; ++cb) xl[((wr * RB + rb) * 8 + cb) * 64 + l] = acc[rb][cb];
            }
            __syncthreads();
            if (wc == 1) return;
        }
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
            const int row = tok[rb];
            if (row < 0) continue;
#pragma unroll
            for (int cb = 0; cb < 8; ++cb) {
                const int col = c0 + cb * 16 + 4 * lg;
                if (col >= N) continue;
                f32x4 v = acc[rb][cb];
                if (pair) {
                    const f32x4 u = xl[((wr * RB + rb) * 8 + cb) * 64 + l];
#pragma unroll
                    for (int i = 0; i < 4; ++i) v[i] = v[i] / (1.f + __expf(-v[i])) * u[i];
                }
                const size_t idx = ((size_t)(row >> 4) * a.h_KS + (col >> 5)) * kFrag +
                                   ((row & 15) + 16 * ((col & 31) >> 3)) * 8 + (col & 7);
                const uint32_t lo = (uint32_t)f2bf(v[0]) | ((uint32_t)f2bf(v[1]) << 16);
                const uint32_t hi = (uint32_t)f2bf(v[2]) | ((uint32_t)f2bf(v[3]) << 16);
                *reinterpret_cast<uint2*>(a.h_dst + idx) = make_uint2(lo, hi);
            }
        }
        return;
    }
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
    // every projection of a launch reads X the same way; row-major X needs
    // an even number of k-steps (pairs share a 128-byte line)
    const bool xrm = a.p[0].x_rowmajor != 0;
    for (int i = 0; i < a.n_proj; ++i)
        if ((a.p[i].x_rowmajor != 0) != xrm || (xrm && (a.p[i].K & 63) != 0)) return hipErrorInvalidValue;
    if (xrm)
        hipLaunchKernelGGL((gemm_big_kernel<kBigRB, true>), dim3(a.total_tiles), dim3(128 * (16 / kBigRB)), 0, s, a);
    else
        hipLaunchKernelGGL((gemm_big_kernel<kBigRB, false>), dim3(a.total_tiles), dim3(128 * (16 / kBigRB)), 0, s, a);
    if (a.total_fix > 0) {
        FwdArgs f = a;
        f.fixup = 1;
        hipLaunchKernelGGL((gemm_big_kernel<kBigRB, false>), dim3(a.total_fix), dim3(128 * (16 / kBigRB)), 0, s, f);
    }
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Medium batches (kDecodeMaxT < T <= kMidMaxT, bf16 base): the base product
// X W_s of Alg. 1 / Alg. 2 with every row of the batch in one tile, so each
// weight fragment is read from HBM once and meets all T rows.
//
// Work item = (projection, 8 NB column blocks, k-range).  Per k-step the RB
// activation fragments (all rows, gathered from the caller's row-major X)
// go from global memory into LDS by DMA, kMidStages k-steps deep, and all
// eight waves read them there; each wave copies its own NB weight fragments
// into LDS the same way, so that every load a k-step waits for is such a
// copy (the wait counts loads in flight, and a load into registers can
// complete ahead of an older copy into LDS).  A wave issues RB NB MFMAs per
// k-step (weight fragment as the A operand: a lane holds 4 consecutive
// columns of one row).  Every item stores its fp32 sum as a partial tile in
// lane order ((wave RB + rb) NB + cb) 64 + lane.  The k-ranges split long-K
// tiles so that the items fill the chip once.
//
// mid_epi_kernel then computes each output: the sum of its partials in
// range order plus the expand of the token's own adapter (steps "Y_adapter
// <- Z B" and "Y <- Y + Y_adapter"), sum_j Z[t, j] B^T[n, j] in fp32 FMAs
// over the token's own ranks only, and one bf16 (or fp32) store.
// ---------------------------------------------------------------------------

constexpr int kMidStages = 4;

// copy 16 bytes per lane (byte offset vo of the buffer) to lane's slot of the
// 1 KB fragment at dst
__device__ __forceinline__ void mid_copy(__amdgpu_buffer_rsrc_t r, u32x4* dst, int vo) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)dst, 16, vo, 0, 0, 0);
}

template <int RB, int NB>
__global__ __launch_bounds__(512) void gemm_mid_kernel(FwdArgs a) {
    constexpr int NW = 8, CPX = RB / NW, D = kMidStages;
    constexpr int SF = RB + NW * NB;          // fragments per stage: activations, then each wave's weights
    static_assert(RB % NW == 0 && D >= 3, "each wave copies RB / 8 fragments per k-step");
    static_assert(D * SF * 1024 <= 160 * 1024, "the stages fit the LDS");
    __shared__ u32x4 lds[D * SF * 64];
    const int w = wave_id(), l = threadIdx.x & 63;
    const int bid = blockIdx.x;
    if (bid >= a.mid_items) return;
    int p = 0;
#pragma unroll
    for (int q = 1; q < kMaxProjs; ++q)
        if (q < a.n_proj && bid >= a.p[q].part_base) p = q;
    const ProjLaunch& P = a.p[p];
    const int S = P.ksplit, item = bid - P.part_base, tile = item / S, split = item - tile * S;
    const int T = a.T, KS = P.K >> 5, nrb = (T + 15) >> 4, ncb = P.N >> 4;
    const int k0 = split * KS / S, NK = (split + 1) * KS / S - k0;

    // activation copies of a k-step: row block w + 8 i, i < CPX, of the tile.
    // Tile rows are positions in rowtok order (tokens grouped by adapter, so
    // the epilogue's consecutive rows share adapters); each lane gathers its
    // row's token through its buffer-load offset, and the copy puts lane l's
    // 16 bytes at byte 16 l of the LDS fragment, so lane l = r + 16 c loads
    // inputs 32 ks + 8 c .. + 7 of row r's token: in the caller's row-major
    // X (k-steps 64 bytes apart; buffer bounds = X's size) or in the packed X
    // (the token's fragment, lane slot (token mod 16) + 16 c; k-steps a
    // fragment apart).  Rows past T repeat a valid token (their sums are
    // never read).
    const bool xrm = P.x_rowmajor != 0;
    const __amdgpu_buffer_rsrc_t rx =
        xrm ? __builtin_amdgcn_make_buffer_rsrc((void*)P.X, 0, T * P.K * 2, kRawBufferWord3)
            : __builtin_amdgcn_make_buffer_rsrc((void*)P.Xp, 0, nrb * KS * 1024, kRawBufferWord3);
    const int xst = xrm ? 64 : 1024;       // bytes from one k-step to the next
    int vo[CPX];
#pragma unroll
    for (int i = 0; i < CPX; ++i) {
        const int pos = min((w + NW * i) * 16 + (l & 15), T - 1);
        const int t = (int)min((unsigned)a.rowtok[pos], (unsigned)(T - 1));
        vo[i] = xrm ? (t * P.K + k0 * 32 + 8 * (l >> 4)) * 2
                    : ((t >> 4) * KS + k0) * 1024 + ((t & 15) + 16 * (l >> 4)) * 16;
    }
    // this wave's weight column blocks (clamped at the projection's edge):
    // copied the same way into the wave's own fragments RB + w NB + c of the
    // stage.  Every load of a turn is then a copy into LDS: a load into
    // registers issued after a copy can complete before it, so a wait that
    // counts outstanding loads over both kinds would not tell that the
    // older copy has landed.
    const __amdgpu_buffer_rsrc_t rw =
        __builtin_amdgcn_make_buffer_rsrc((void*)P.W, 0, ncb * KS * 1024, kRawBufferWord3);
    int wo[NB];
#pragma unroll
    for (int c = 0; c < NB; ++c) wo[c] = (int)frag_index(min((tile * NW + w) * NB + c, ncb - 1), k0, KS) * 2 + l * 16;

    // one pipeline turn: the activations and weights of k-step ks into LDS
    // stage d.  Past the range the last k-step is loaded again, so every
    // turn issues the same number of copies and the wait counts below are
    // exact.
    auto issue = [&](int ks, int d) __attribute__((always_inline)) {
        const int kk = min(ks, NK - 1);
        u32x4* stg = lds + d * SF * 64;
#pragma unroll
        for (int i = 0; i < CPX; ++i)
            mid_copy(rx, stg + (w + NW * i) * 64, vo[i] + kk * xst);
#pragma unroll
        for (int c = 0; c < NB; ++c) mid_copy(rw, stg + (RB + w * NB + c) * 64, wo[c] + kk * 1024);
    };

    f32x4 acc[RB][NB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int c = 0; c < NB; ++c) acc[rb][c] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int d = 0; d < D - 1; ++d) issue(d, d);

    // k-step ks uses stage u = ks mod D.  Its copies are complete once at
    // most the D - 2 later turns are in flight; the barrier makes every
    // wave's copies visible and ends every wave's reads of k-step ks - 1,
    // whose stage the next turn refills.
    auto step = [&](int ks, int u) __attribute__((always_inline)) {
        big_wait_barrier<(D - 2) * (CPX + NB)>();
        issue(ks + D - 1, (u + D - 1) % D);
        const u32x4* stg = lds + u * SF * 64;
        u32x4 wv[NB];
#pragma unroll
        for (int c = 0; c < NB; ++c) wv[c] = stg[(RB + w * NB + c) * 64 + l];
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
            const u32x4 x = stg[rb * 64 + l];
#pragma unroll
            for (int c = 0; c < NB; ++c) acc[rb][c] = mfma(wv[c], x, acc[rb][c]);
        }
    };
    int ks = 0;
    for (; ks + D <= NK; ks += D) {
#pragma unroll
        for (int u = 0; u < D; ++u) step(ks + u, u);
    }
#pragma unroll
    for (int u = 0; u < D; ++u)
        if (ks + u < NK) step(ks + u, u);
    // no copy into LDS may still be in flight when the workgroup ends
    big_wait_barrier<0>();

    f32x4* dst = reinterpret_cast<f32x4*>(a.bigpart) + (size_t)(P.part_base + item) * (kBigPartElems / 4) +
                 (size_t)w * RB * NB * 64 + l;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
        if (rb < nrb)
#pragma unroll
            for (int c = 0; c < NB; ++c) dst[(rb * NB + c) * 64] = acc[rb][c];
}

// Epilogue workgroups: 256 threads over one 64-column tile; thread (t, g)
// computes the outputs of row t in columns CPT g .. CPT g + CPT - 1, so a
// workgroup covers 256 CPT / 64 rows.  Four columns per thread keep the
// registers (and so the resident waves) of a thread's loads in flight low.
constexpr int kMidEpiCols = 4;    // columns per thread
constexpr int kMidEpiSeg = 2;     // partials per output loaded before the first sum

// acc[c] += sum_e z_e B^T[c][e] over 8 ranks, z_e = hi + lo of the bf16 pair
template <int CPT>
__device__ __forceinline__ void fma_ranks8(float (&acc)[CPT], const u32x4 (&b)[CPT], const u32x4& zh,
                                           const u32x4& zl) {
    const uint32_t h[4] = {zh.x, zh.y, zh.z, zh.w}, o[4] = {zl.x, zl.y, zl.z, zl.w};
    float z[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        z[2 * e] = __uint_as_float(h[e] << 16) + __uint_as_float(o[e] << 16);
        z[2 * e + 1] = __uint_as_float(h[e] & 0xffff0000u) + __uint_as_float(o[e] & 0xffff0000u);
    }
#pragma unroll
    for (int c = 0; c < CPT; ++c) {
        const uint32_t q[4] = {b[c].x, b[c].y, b[c].z, b[c].w};
        float sum = 0.f;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            sum = fmaf(z[2 * e], __uint_as_float(q[e] << 16), sum);
            sum = fmaf(z[2 * e + 1], __uint_as_float(q[e] & 0xffff0000u), sum);
        }
        acc[c] += sum;
    }
}

// Workgroup rows and their LDS: RPW rows x 64 columns of B^T ranks 0..15.
template <int CPT>
struct MidEpiLds {
    static constexpr int TPR = 64 / CPT, RPW = 256 / TPR;   // threads per row, rows per workgroup
    u32x4 bl[RPW * 64 * 2];
    int rinfo[RPW];
};

// The outputs of row position pos (rowtok order; token tt) in columns
// col .. col + CPT - 1 of 64-column tile `local` of projection P: the sum of
// its partials in range order plus the expand of the token's own adapter,
// in fp32.  Every thread of the workgroup calls it (it holds barriers).
template <int CPT>
__device__ __forceinline__ void mid_epi_sum(const FwdArgs& a, const ProjLaunch& P, int local, int pos, int col,
                                            MidEpiLds<CPT>& sh, float (&acc)[CPT]) {
    constexpr int TPR = MidEpiLds<CPT>::TPR, RPW = MidEpiLds<CPT>::RPW, NQ = CPT / 4;
    const int T = a.T, N = P.N;
    const int pp = min(pos, T - 1), cc = min(col, N - CPT);
    // the row's adapter (slot and rank, from the plan's row table) and token,
    // loaded before the partials so that waiting for them leaves the
    // partials in flight
    const int info = a.rowslot[pp];
    // (clamped: a bad entry can cost a wrong row, never an access past Z or out)
    const int tt = (int)min((unsigned)a.rowtok[pp], (unsigned)(T - 1));

    // partials: columns cc + 4 q .. + 3 of row pp are lane ln + 16 q of block
    // (pp / 16, cc / 16) of wave wq of column tile tc
    const int mnb = a.mid_nb, S = P.ksplit, rbg = pp >> 4, cbg = cc >> 4;
    const int tc = cbg / (8 * mnb), wq = (cbg - tc * 8 * mnb) / mnb, cq = cbg - tc * 8 * mnb - wq * mnb;
    const int ln = (pp & 15) + 16 * ((cc & 15) >> 2);
    const f32x4* src = reinterpret_cast<const f32x4*>(a.bigpart) + (size_t)(P.part_base + tc * S) * (kBigPartElems / 4) +
                       ((size_t)(wq * a.mid_rb + rbg) * mnb + cq) * 64 + ln;
    f32x4 y[kMidEpiSeg][NQ];
#pragma unroll
    for (int j = 0; j < kMidEpiSeg; ++j) {
        const size_t o = (size_t)min(j, S - 1) * (kBigPartElems / 4);
#pragma unroll
        for (int q = 0; q < NQ; ++q) y[j][q] = src[o + 16 * q];
    }

    // the token's own adapter: ranks 0..15 of B^T and of Z, loaded without a
    // branch (a half the rank does not have reads ranks 0..7 again, unused)
    // (clamped: a bad entry can cost a wrong sum, never an access past the pool)
    const int v = info >= 0 ? min(info & 0xffff, a.max_slots - 1) : -1;
    const int r8s = info >= 0 ? min(info >> 16, a.r8max) : 0;
    int sig = 0;
#pragma unroll
    for (int q = 1; q < kMaxSlices; ++q)
        if (q < P.n_slices && cc >= P.slice_col[q]) sig = q;
    const uint16_t* bb = a.pool + (size_t)max(v, 0) * a.slot_stride + P.b_off + (size_t)cc * r8s;
    const uint16_t* zp = P.Z + (size_t)tt * P.zs + sig * a.r8max;
    u32x4 zh[2], zl[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int ho = 8 * h < r8s ? 8 * h : 0;
        zh[h] = ld16(zp + ho);
        zl[h] = ld16(zp + ho + P.zplane);
    }

    // Ranks 0..15 of each row's B^T slice (64 columns of the tile) through
    // LDS: the workgroup loads the RPW slices with 16-byte loads in which
    // consecutive lanes read consecutive (column, rank half) pieces, so a wave
    // instruction covers contiguous bytes, where each thread reading its own
    // columns straight from HBM would touch a cache line per lane.  A slice
    // is stored column-interleaved (column c in slot (c mod CPT) 64 / CPT +
    // c / CPT), so the threads of a row reading one of their columns read
    // consecutive 32-byte slots (two-way bank conflicts; a padded slot would
    // avoid them but the extra LDS costs more in resident workgroups).
    constexpr int SLOT = 2;                      // u32x4 per column slot: rank halves 0, 1
    const int rl = threadIdx.x / TPR;            // this thread's row in the workgroup
    __syncthreads();                             // a previous call's readers are done
    if (threadIdx.x % TPR == 0) sh.rinfo[rl] = info;
    __syncthreads();
    const int tile_c0 = local * 64;
#pragma unroll
    for (int k = 0; k < RPW * 128 / 256; ++k) {
        const int idx = k * 256 + threadIdx.x, row = idx >> 7, pc = idx & 127, c = pc >> 1, h = pc & 1;
        const int inf = sh.rinfo[row];
        const int vs = inf >= 0 ? min(inf & 0xffff, a.max_slots - 1) : 0;
        const int rs = inf >= 0 ? min(inf >> 16, a.r8max) : 0;
        // columns past N and halves past the rank read a valid piece, unused
        const int col_c = min(tile_c0 + c, N - 1), hh = 8 * h < rs ? 8 * h : 0;
        const u32x4 piece = ld16(a.pool + (size_t)vs * a.slot_stride + P.b_off + (size_t)col_c * rs + hh);
        sh.bl[(row * 64 + (c % CPT) * (64 / CPT) + c / CPT) * SLOT + h] = piece;
    }
    __syncthreads();
    u32x4 bq[2][CPT];
    {
        const int g = (threadIdx.x % TPR) - (col - cc) / CPT;   // column group of cc in the tile
#pragma unroll
        for (int c = 0; c < CPT; ++c)
#pragma unroll
            for (int h = 0; h < 2; ++h) bq[h][c] = sh.bl[(rl * 64 + c * (64 / CPT) + g) * SLOT + h];
    }

#pragma unroll
    for (int c = 0; c < CPT; ++c) acc[c] = 0.f;
#pragma unroll
    for (int j = 0; j < kMidEpiSeg; ++j)
        if (j < S) {
#pragma unroll
            for (int q = 0; q < NQ; ++q)
#pragma unroll
                for (int i = 0; i < 4; ++i) acc[4 * q + i] += y[j][q][i];
        }
    for (int j = kMidEpiSeg; j < S; ++j) {
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const f32x4 u = src[(size_t)j * (kBigPartElems / 4) + 16 * q];
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[4 * q + i] += u[i];
        }
    }
#pragma unroll
    for (int h = 0; h < 2; ++h)
        if (8 * h < r8s) fma_ranks8<CPT>(acc, bq[h], zh[h], zl[h]);
    // ranks 16 and up, 8 at a time
    for (int j0 = 16; j0 < r8s; j0 += 8) {
        u32x4 br[CPT];
#pragma unroll
        for (int c = 0; c < CPT; ++c) br[c] = ld16(bb + (size_t)c * r8s + j0);
        fma_ranks8<CPT>(acc, br, ld16(zp + j0), ld16(zp + j0 + P.zplane));
    }
}

template <int CPT>
__global__ __launch_bounds__(256) void mid_epi_kernel(FwdArgs a) {
    static_assert(CPT == 4 || CPT == 8, "one or two 4-column lanes of a partial block");
    constexpr int TPR = MidEpiLds<CPT>::TPR, RPW = MidEpiLds<CPT>::RPW, NQ = CPT / 4;
    __shared__ MidEpiLds<CPT> sh;
    const int tile = blockIdx.x;
    int p = 0;
#pragma unroll
    for (int q = 1; q < kMaxProjs; ++q)
        if (q < a.n_proj && tile >= a.p[q].col_base) p = q;
    const ProjLaunch& P = a.p[p];
    const int T = a.T, N = P.N;
    // rows are positions in rowtok order (those of the main launch's tile)
    const int pos = blockIdx.y * RPW + threadIdx.x / TPR;
    const int col = (tile - P.col_base) * 64 + (threadIdx.x % TPR) * CPT;
    // threads past the last row or column compute on clamped indices and
    // store nothing (every load is issued without waiting on a branch)
    const bool live = pos < T && col < N;
    const int tt = (int)min((unsigned)a.rowtok[min(pos, T - 1)], (unsigned)(T - 1));
    float acc[CPT];
    mid_epi_sum<CPT>(a, P, tile - P.col_base, pos, col, sh, acc);
    if (a.mlp_act == BDLORA_ACT_SILU_MUL) {
        // gate's tiles only: up (projection p + 1) for the same outputs
        float up[CPT];
        mid_epi_sum<CPT>(a, a.p[p + 1], tile - P.col_base, pos, col, sh, up);
#pragma unroll
        for (int c = 0; c < CPT; ++c) acc[c] = acc[c] / (1.f + __expf(-acc[c])) * up[c];
    }
    if (!live) return;
    if (a.mlp_act >= 0) {
        // the MLP intermediate H in bf16 in the second projection's input
        // layout (token tt, columns col ..): CPT / 4 pieces of 4 contiguous
        // elements
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int c = col + 4 * q;
            const size_t idx = ((size_t)(tt >> 4) * a.h_KS + (c >> 5)) * kFrag + ((tt & 15) + 16 * ((c & 31) >> 3)) * 8 +
                               (c & 7);
            const uint32_t lo = (uint32_t)f2bf(acc[4 * q]) | ((uint32_t)f2bf(acc[4 * q + 1]) << 16);
            const uint32_t hi = (uint32_t)f2bf(acc[4 * q + 2]) | ((uint32_t)f2bf(acc[4 * q + 3]) << 16);
            *reinterpret_cast<uint2*>(a.h_dst + idx) = make_uint2(lo, hi);
        }
        return;
    }
    if (P.out_f32) {
        float* o = P.out_f32 + (size_t)tt * N + col;
#pragma unroll
        for (int q = 0; q < NQ; ++q)
            *reinterpret_cast<float4*>(o + 4 * q) = make_float4(acc[4 * q], acc[4 * q + 1], acc[4 * q + 2], acc[4 * q + 3]);
    } else {
        uint32_t w[CPT / 2];
#pragma unroll
        for (int c = 0; c < CPT / 2; ++c) w[c] = (uint32_t)f2bf(acc[2 * c]) | ((uint32_t)f2bf(acc[2 * c + 1]) << 16);
        uint16_t* o = P.out + (size_t)tt * N + col;
        if constexpr (CPT == 8)
            *reinterpret_cast<u32x4*>(o) = u32x4{w[0], w[1], w[2], w[3]};
        else
            *reinterpret_cast<uint2*>(o) = make_uint2(w[0], w[1]);
    }
}

hipError_t launch_gemm_mid(const FwdArgs& a, hipStream_t s) {
    if (a.mid_items <= 0) return hipSuccess;
    if (a.T <= 0 || a.T > a.mid_rb * 16 || a.mid_rb * a.mid_nb * 2048 > kBigPartElems || !a.rowtok)
        return hipErrorInvalidValue;
    bool ok = false;
#define BDL_MID_CASE(R, NN)                                                                     \
    if (a.mid_rb == R && a.mid_nb == NN) {                                                      \
        hipLaunchKernelGGL((gemm_mid_kernel<R, NN>), dim3(a.mid_items), dim3(512), 0, s, a);    \
        ok = true;                                                                              \
    }
    BDL_MID_CASE(8, 1) BDL_MID_CASE(8, 2) BDL_MID_CASE(16, 1) BDL_MID_CASE(16, 2)
#undef BDL_MID_CASE
    if (!ok) return hipErrorInvalidValue;
    return hipGetLastError();
}

hipError_t launch_mid_epi(const FwdArgs& a, hipStream_t s) {
    if (a.mid_items <= 0) return hipSuccess;
    if (a.T <= 0 || a.mid_col_tiles <= 0 || !a.rowtok || !a.rowslot) return hipErrorInvalidValue;
    constexpr int rows = 256 / (64 / kMidEpiCols);   // rows per workgroup
    hipLaunchKernelGGL(mid_epi_kernel<kMidEpiCols>, dim3(a.mid_col_tiles, (a.T + rows - 1) / rows), dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace bdl
