// Decode path (batches of at most kDecodeMaxT tokens): two launches after
// the prep launch (plan + activation packing); small batches (at most 32
// tokens, by the host's rule) skip the prep launch (the main launch plans
// the batch in every wave and gathers the caller's X).
//
//  dec_main_kernel -- one split-K GEMM of the packed activations X [T x K]
//                     against a virtual column list per projection: the
//                     16-column blocks of W_s, then the blocks of A^T_cat of
//                     every adapter the batch uses.  So one pass streams the
//                     base weight once (step "Y <- X W" of Alg. 1 / Alg. 2)
//                     and every used adapter's A once (step "Z <- X A"),
//                     computing Z for all tokens against all used adapters;
//                     the epilogue keeps each token's own.  Work is counted in
//                     units of one block times one 32-wide k-step; consecutive
//                     blocks form groups of 4, and workgroup b takes the
//                     k-steps whose first unit lies in [b U / G, (b+1) U / G),
//                     so all G workgroups stream the same number of bytes.
//                     Workgroups are 4 waves that split the group's
//                     blocks and the k-range (see dec_flush).
//                     Each (group, workgroup) pair writes one fp32 partial
//                     tile to slot g + b (injective: along the unit order both
//                     indices only grow).
//  dec_epi_kernel  -- per 64-column output tile, all tokens:
//                     out[t, n] = sum of the tile's partials
//                                 + scale * sum_j Z[t, j] B^T[n, j]
//                     with Z[t, :] summed from the partials of the token's own
//                     adapter (steps "Y_adapter <- Z B", "Y <- Y + Y_adapter"),
//                     in fp32, one bf16 store per output.
#include "bdl_device.h"

namespace bdl {

constexpr int kDecStages = 2;

// Position of projection p in the unit and group orders.  The column lists
// hold act_max adapter positions (the host's bound on the number of adapters
// a batch uses, so the schedule is known before the plan is); positions at
// or past the batch's count n_act are skipped.
struct ProjPos {
    unsigned ub;    // first unit (the host keeps U * G below 2^32)
    int gb;         // first group
    int nb;         // virtual blocks
    int KS;         // k-steps
};

__device__ __forceinline__ ProjPos dec_pos(const DecArgs& a, int p) {
    return ProjPos{a.sub[p], a.sgb[p], a.snb[p], a.sks[p]};
}

// workgroup whose unit range holds unit u: largest b with floor(b U / G) <= u
__device__ __forceinline__ int dec_wg_of(unsigned u, unsigned U, int G) {
    return (int)(((u + 1) * (unsigned)G - 1) / U);
}

// A segment: the k-steps [k0, k1) of group gl of projection p that one
// workgroup owns (its unit range cut at group ends).  Everything here is
// uniform over the workgroup.
struct DecSeg {
    int p;
    ProjPos pp;
    int gl;           // group within the projection
    unsigned goff;    // first unit of the group
    int wdt;          // blocks in the group (4, fewer at a projection's end)
    int k0, k1;
    bool valid;
    int dmask;        // bit j: block j of the group holds data for this batch
};

// Which of the blocks 4 gl .. 4 gl + wdt - 1 of projection P's column list
// hold data for this batch (bit j for block 4 gl + j): weight blocks always;
// adapter block v (position v / nbA, block v mod nbA of it) when its
// position is an adapter in use (below n_act) and the block lies within that
// adapter's own rank (lane i of gr holds the padded rank of the i-th adapter
// in use), so a rank-8 adapter in a pool sized for rank 64 streams its own
// blocks only.  One division per group; the positions advance by counting.
__device__ __forceinline__ int dec_group_mask(const DecProj& P, int gl, int wdt, int n_act, int gr) {
    const int v0 = 4 * gl - P.nWb;
    if (v0 + wdt <= 0) return (1 << wdt) - 1;        // weight blocks only
    int ai = v0 > 0 ? v0 / P.nbA : 0, c = v0 > 0 ? v0 - ai * P.nbA : v0;
    int m = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        if (j < wdt) {
            if (c < 0) {
                m |= 1 << j;                           // a weight block
            } else if (ai < n_act && c < ((P.n_slices * __builtin_amdgcn_readlane(gr, ai) + 15) >> 4)) {
                m |= 1 << j;
            }
        }
        if (++c >= P.nbA && c >= 0) {
            c = 0;
            ++ai;
        }
    }
    return m;
}

// cut the segment that starts at k-step g.k0 of the current group, moving to
// the next group (and projection) when that group is used up; groups with no
// weight block and no adapter block holding data are skipped.  n_act and the
// ranks arrive in vector registers (lane-uniform / per lane) and are read
// only for adapter groups, so weight segments never wait for them.
__device__ __forceinline__ void dec_cut(const DecArgs& a, int n_act_v, int gr, unsigned se, DecSeg& g) {
    for (;;) {
        if (g.k0 >= g.pp.KS) {
            if (++g.gl >= ((g.pp.nb + 3) >> 2)) {
                if (++g.p >= a.n_proj) {
                    g.valid = false;
                    return;
                }
                g.pp = dec_pos(a, g.p);
                g.gl = 0;
            }
            g.goff = g.pp.ub + 4u * g.gl * g.pp.KS;
            g.wdt = min(4, g.pp.nb - 4 * g.gl);
            g.k0 = 0;
            if (g.goff >= se) {
                g.valid = false;
                return;
            }
        }
        g.k1 = (int)min((unsigned)g.pp.KS, (se - g.goff + g.wdt - 1) / (unsigned)g.wdt);
        g.valid = g.k1 > g.k0;
        if (!g.valid) return;
        if (4 * g.gl + g.wdt <= a.p[g.p].nWb) {
            g.dmask = (1 << g.wdt) - 1;                // weight blocks only
            return;
        }
        g.dmask = dec_group_mask(a.p[g.p], g.gl, g.wdt, __builtin_amdgcn_readfirstlane(n_act_v), gr);
        if (g.dmask) return;
        g.k0 = g.pp.KS;
    }
}

// first segment of the unit range [sb, se): the group holding unit sb, from
// its first k-step starting at or after sb
__device__ __forceinline__ DecSeg dec_first(const DecArgs& a, int n_act_v, int gr, unsigned sb, unsigned se) {
    DecSeg g;
    g.p = 0;
#pragma unroll
    for (int q = 1; q < kMaxProjs; ++q)
        if (q < a.n_proj && sb >= a.sub[q]) g.p = q;
    g.pp = dec_pos(a, g.p);
    g.gl = min((int)((sb - g.pp.ub) / (4u * g.pp.KS)), ((g.pp.nb + 3) >> 2) - 1);
    g.goff = g.pp.ub + 4u * g.gl * g.pp.KS;
    g.wdt = min(4, g.pp.nb - 4 * g.gl);
    g.k0 = (int)((sb - g.goff + g.wdt - 1) / (unsigned)g.wdt);
    dec_cut(a, n_act_v, gr, se, g);
    return g;
}

__device__ __forceinline__ void dec_next(const DecArgs& a, int n_act_v, int gr, unsigned se, DecSeg& g) {
    g.k0 = g.k1;
    dec_cut(a, n_act_v, gr, se, g);
}

// The k-steps of a segment that K-part kq of NKQ handles: [*kw, *kw + items).
template <int NKQ>
__device__ __forceinline__ int dec_items(const DecSeg& g, int kq, int* kw) {
    const int n = g.k1 - g.k0, q = n / NKQ, r = n - q * NKQ;
    *kw = g.k0 + kq * q + min(kq, r);
    return q + (kq < r ? 1 : 0);
}

// element pointer of k-step 0 of virtual block vb of projection P; lane i of
// gs holds the slot of the i-th adapter in use (entries at or past n_act are
// not written by the plan).  Positions at or past n_act (in a group with a
// weight block or a used adapter) read slot 0's factor, unused: that slot
// always exists, whatever the table holds.
__device__ __forceinline__ const uint16_t* dec_block(const DecArgs& a, const DecProj& P, int vb, int KS, int gs,
                                                     int n_act_v) {
    if (vb < P.nWb) return P.W + frag_index(vb, 0, KS);
    const int ai = (vb - P.nWb) / P.nbA, c = vb - P.nWb - ai * P.nbA;
    const bool used = ai < __builtin_amdgcn_readfirstlane(n_act_v);
    const int slot = used ? __builtin_amdgcn_readlane(gs, used ? ai : 0) : 0;
    return a.pool + (size_t)slot * a.slot_stride + P.a_off + frag_index(c, 0, KS);
}

// The batch's plan, computed by a wave of the main launch (lane t holds
// token t; T <= 64), with the prep launch's decode plan's results: ids
// checked against the loaded slots, the adapters in use in ascending slot
// order ("groups"; at most act_max of them: any past that bound, possible
// only when a captured forward replays after more adapters were loaded, are
// treated as none and raise the error flag), each token's group.  Lane g
// gets the slot and padded rank of group g (0 from the count on); the count
// is returned.  Pools of at most 64 slots keep the slot tables in lanes (one
// load round trip) and send each slot in use to the lane of its rank among
// them; larger pools look the tables up per token and take the smallest
// remaining slot per pass.  With store set the wave also writes the
// per-token tables the epilogue reads (vid, tr8, tgrp), the group tables and
// count, and the error flag.
__device__ __forceinline__ int dec_plan(const DecArgs& a, bool store, int* gs_out, int* gr_out) {
    const int l = threadIdx.x & 63;
    const bool in = l < a.T;
    const bool small = a.max_slots <= 64;
    const int lt = small && l < a.max_slots ? a.loaded[l] : 0;
    const int rt = small && l < a.max_slots ? a.r8[l] : 0;
    int id = -1;
    if (a.ids) {
        id = in ? a.ids[l] : -1;
    } else {
        // segments in token order: the last one starting at or before t
        for (int i = 0; i < a.n_seg; ++i)
            if (l >= a.seg_start[i]) id = a.seg_slot[i];
        if (!in) id = -1;
    }
    const bool in_range = id >= 0 && id < a.max_slots;
    int ld, r8v;
    if (small) {
        ld = __shfl(lt, in_range ? id : 0);
        r8v = __shfl(rt, in_range ? id : 0);
        if (!in_range) ld = r8v = 0;
    } else {
        ld = in_range ? a.loaded[id] : 0;
        r8v = in_range ? a.r8[id] : 0;
    }
    bool ok = in_range && ld != 0;
    bool bad = __ballot(in && !ok && id != -1) != 0ull;
    int g = 0, mine = -1, gs = 0, gr = 0;
    const int v = ok ? id : -1;
    if (small) {
        const unsigned long long bit = ok ? 1ull << v : 0ull;
        const unsigned long long used =
            (unsigned long long)wave_or((unsigned)bit) | ((unsigned long long)wave_or((unsigned)(bit >> 32)) << 32);
        g = __popcll(used);
        // lane l holds slot l: a slot in use goes to the lane of its rank
        // among them, the other lanes to the lanes from g on (together a
        // permutation of the 64 lanes)
        const int below = __popcll(used & ((1ull << l) - 1ull));
        const int to = ((used >> l) & 1ull) ? below : g + (l - below);
        gs = __builtin_amdgcn_ds_permute(to * 4, l);
        gr = __builtin_amdgcn_ds_permute(to * 4, rt);
        if (ok) mine = __popcll(used & (bit - 1ull));
    } else {
        unsigned long long rem = __ballot(ok);
        while (rem) {
            const int m = wave_min(((rem >> l) & 1ull) ? v : 0x7fffffff);
            const bool eq = ok && v == m;
            if (eq) mine = g;
            // slot m's rank: held by every lane whose token uses it
            const int rm = __builtin_amdgcn_readlane(r8v, __ffsll((long long)__ballot(eq)) - 1);
            if (l == g) {
                gs = m;
                gr = rm;
            }
            ++g;
            rem &= ~__ballot(eq);
        }
    }
    if (g > a.act_max) {
        const bool over = ok && mine >= a.act_max;
        bad = bad || __ballot(over) != 0ull;
        if (over) {
            ok = false;
            mine = -1;
        }
        g = a.act_max;
    }
    if (l >= g) gs = gr = 0;
    if (store) {
        if (in) {
            a.vid[l] = ok ? v : -1;
            a.tr8[l] = ok ? r8v : 0;
            a.tgrp[l] = mine;
        }
        if (l < g) {
            a.gslot[l] = gs;
            a.gr8[l] = gr;
        }
        if (l == 0) {
            a.meta[0] = g;
            a.meta[1] = 0;
            if (bad) atomicOr(a.err, 1);
        }
    }
    *gs_out = gs;
    *gr_out = gr;
    return g;
}

// Four waves per workgroup as 4 / NB column groups x NB parts of the
// segment's k-range; a wave takes NB of the group's 4 blocks (4 for bf16
// weights, 2 in launches with an INT4 base, whose unpacking needs the
// registers): per k-step it loads MB activation fragments and NB weight
// fragments and issues NB MB MFMAs, so every activation fragment it loads
// serves NB blocks.  At the end of a segment the K-parts meet in LDS; all
// 256 threads add them in a fixed order and store the group's fp32 partial
// (rows < T, the group's wdt blocks) as 16-byte chunks.
constexpr int kDecWaves = 4;
constexpr int kDecThreads = 64 * kDecWaves;
constexpr int kRedLd = 68;    // LDS row stride (floats): 4 rows apart land 16 banks apart

template <int MB, int NB>
__device__ __forceinline__ void dec_flush(const DecArgs& a, const DecSeg& g, f32x4 (&acc)[MB][NB], float* red, int b) {
    constexpr int REG = MB * 16 * kRedLd, NCG = 4 / NB, NKQ = kDecWaves / NCG;
    const int w = wave_id(), l = threadIdx.x & 63, cg = w % NCG, kq = w / NCG;
    __syncthreads();                          // the previous segment's readers are done
    float* reg = red + kq * REG + cg * NB * 16 + (l & 15);
#pragma unroll
    for (int rb = 0; rb < MB; ++rb)
#pragma unroll
        for (int cb = 0; cb < NB; ++cb)
#pragma unroll
            for (int i = 0; i < 4; ++i) reg[(rb * 16 + 4 * (l >> 4) + i) * kRedLd + cb * 16] = acc[rb][cb][i];
#pragma unroll
    for (int rb = 0; rb < MB; ++rb)
#pragma unroll
        for (int cb = 0; cb < NB; ++cb) acc[rb][cb] = f32x4{0.f, 0.f, 0.f, 0.f};
    __syncthreads();
    float* dst = a.part + (size_t)min(g.pp.gb + g.gl + b, a.part_slots - 1) * kPartElems;
    const int nc4 = g.wdt * 4;
#pragma unroll
    for (int j = 0; j < MB; ++j) {
        const int c = threadIdx.x + j * kDecThreads;   // MB * 16 rows x 16 four-column chunks
        const int row = c >> 4, c4 = c & 15;
        if (row < a.T && c4 < nc4) {
            const float* src = red + row * kRedLd + c4 * 4;
            float4 v = *reinterpret_cast<const float4*>(src);
#pragma unroll
            for (int k = 1; k < NKQ; ++k) {
                const float4 u = *reinterpret_cast<const float4*>(src + k * REG);
                v.x += u.x; v.y += u.y; v.z += u.z; v.w += u.w;
            }
            *reinterpret_cast<float4*>(dst + row * 64 + c4 * 4) = v;
        }
    }
}

template <int MB, int NB>
__device__ __forceinline__ void mma_nb(f32x4 (&acc)[MB][NB], const u32x4 (&xa)[MB], const u32x4 (&wb)[NB]) {
#pragma unroll
    for (int rb = 0; rb < MB; ++rb)
#pragma unroll
        for (int cb = 0; cb < NB; ++cb) acc[rb][cb] = mfma(xa[rb], wb[cb], acc[rb][cb]);
}

// INT4 base blocks: wb[cb].x holds the lane's word, wb[cb].y the scale bits
template <int MB, int NB>
__device__ __forceinline__ void mma_nb_int4(f32x4 (&acc)[MB][NB], const u32x4 (&xa)[MB], const u32x4 (&wb)[NB]) {
    uint32_t q[NB], sc[NB];
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) {
        q[cb] = wb[cb].x;
        sc[cb] = wb[cb].y;
    }
    mma_int4_kstep<MB, NB>(acc, xa, q, sc);
}

// The workgroup's segments run through one load pipeline of kDecStages
// k-steps per wave: a load cursor walks the wave's k-steps segment after
// segment that many k-steps ahead of the compute loop, so the loads of the
// next segment are in flight while the current one is reduced and stored.
// Each segment's k-steps are padded to a multiple of kDecStages (the padding
// repeats the last load), so every segment starts on the first stage and
// each load's only consumer is one pipeline turn later.  Operand bases are
// wave-uniform (scalar registers); per k-step only the lanes' byte offset
// moves, so the steady state costs one vector add per k-step.
//
// Q4: some projection of the launch has an INT4 base (the kernel then handles
// both operand types; without it the INT4 code is compiled out).  XR (one
// or two row blocks): every wave plans the batch itself and the activations
// are gathered from the caller's row-major X, so no prep launch runs before.
template <int MB, bool Q4, bool XR>
__global__ __launch_bounds__(kDecThreads) __attribute__((amdgpu_waves_per_eu(2))) void dec_main_kernel(DecArgs a) {
    static_assert(!XR || MB <= 2, "row-major activations: at most two row blocks");
    constexpr int NB = Q4 ? 2 : 4, NCG = 4 / NB, NKQ = kDecWaves / NCG;
    __shared__ float red[NKQ * MB * 16 * kRedLd];
    const int w = wave_id(), l = threadIdx.x & 63, cg = w % NCG, kq = w / NCG;
    const int G = gridDim.x, b = blockIdx.x;
    const unsigned U = a.units;               // the host launches with U >= 4 G
    const unsigned sb = (unsigned)b * U / (unsigned)G, se = (unsigned)(b + 1) * U / (unsigned)G;
    // The plan's outputs (n_act, the slots of the adapters in use; at most
    // kDecodeMaxT = 64 of them) are read with vector loads issued here and
    // waited for only where an adapter segment first needs them, so the base
    // weight's loads start without waiting for the plan; with XR every wave
    // computes them (one load round trip for pools of at most 64 slots).
    int gs, gr, n_act_v;
    if constexpr (XR) {
        n_act_v = dec_plan(a, b == 0 && w == 0, &gs, &gr);
    } else {
        gs = l < a.act_max ? a.gslot[l] : 0;
        gr = l < a.act_max ? a.gr8[l] : 0;
        n_act_v = __builtin_amdgcn_raw_buffer_load_b32(
            __builtin_amdgcn_make_buffer_rsrc((void*)a.meta, 0, 4, kRawBufferWord3), 0, 0, 0);
    }
    DecSeg cs = dec_first(a, n_act_v, gr, sb, se);
    if (!cs.valid) return;

    // load cursor: segment, this wave's first k-step and load count in it
    // (padded), loads left; operand bases (uniform)
    DecSeg ls = cs;
    int lkw = 0, lrem = 0, lk = 0, llast = 0;
    const char* xb[MB];                       // activation row blocks (bytes, k-step 0)
    const char* wbp[NB];                      // this wave's blocks (bytes, k-step 0)
    const char* sbp[NB];                      // INT4 blocks: their scales (bytes, group 0)
    bool lq = false;                          // the loader's segment streams INT4 base blocks
#pragma unroll
    for (int c = 0; c < NB; ++c) wbp[c] = sbp[c] = nullptr;
#pragma unroll
    for (int rb = 0; rb < MB; ++rb) xb[rb] = nullptr;
    auto point = [&]() __attribute__((always_inline)) {
        const DecProj& P = a.p[ls.p];
        const int KS = ls.pp.KS;
        if constexpr (XR) {
            // the caller's row-major X: lane (r, c) of row block rb reads
            // inputs 32 ks + 8 c .. + 7 of token 16 rb + r (tokens past T
            // read token T - 1 again; their sums are never read)
#pragma unroll
            for (int rb = 0; rb < MB; ++rb)
                xb[rb] = reinterpret_cast<const char*>(P.X + (size_t)min(16 * rb + (l & 15), a.T - 1) * P.K) +
                         16 * (l >> 4);
        } else {
#pragma unroll
            for (int rb = 0; rb < MB; ++rb) xb[rb] = reinterpret_cast<const char*>(P.Xp + frag_index(rb, 0, KS));
        }
        lq = Q4 && P.Ws && 4 * ls.gl < P.nWb;
        const size_t qs = (size_t)KS * kInt4FragBytes, ss = (size_t)(KS / kInt4Group) * 32;
        // blocks that hold no data for this batch (past an adapter's own rank,
        // or an adapter position not in use) load the group's first block
        // that does instead: the same bytes, served by the caches, so only
        // data blocks cost HBM traffic; their sums are never read.  (The
        // segment's group passed dec_cut, so such a block exists; groups of
        // INT4 weight blocks are never mixed with adapter blocks.)
        const int vbf = 4 * ls.gl + __builtin_ctz((unsigned)ls.dmask | 16u);
#pragma unroll
        for (int c = 0; c < NB; ++c) {
            const int jc = min(cg * NB + c, ls.wdt - 1);
            const int vb = (ls.dmask >> jc) & 1 ? 4 * ls.gl + jc : vbf;
            // both candidates are formed and one is selected (no branch: the
            // bases stay in registers)
            const char* wq = reinterpret_cast<const char*>(P.W) + vb * qs;
            const char* wf = reinterpret_cast<const char*>(dec_block(a, P, vb, KS, gs, n_act_v));
            wbp[c] = lq ? wq : wf;
            sbp[c] = lq ? reinterpret_cast<const char*>(P.Ws) + vb * ss : reinterpret_cast<const char*>(P.Ws);
        }
    };
    // Move the cursor to the next segment in which this wave has k-steps.
    // The bases and [lk, llast] always describe k-steps of a valid segment:
    // past the last segment the cursor stays on the last one it pointed at,
    // so the loads that fill the pipeline's tail repeat a valid address.
    auto advance = [&]() __attribute__((always_inline)) {
        while (lrem == 0) {
            dec_next(a, n_act_v, gr, se, ls);
            if (!ls.valid) return;
            const int n = dec_items<NKQ>(ls, kq, &lkw);
            if (n > 0) {
                lrem = (n + kDecStages - 1) / kDecStages * kDecStages;
                lk = lkw;
                llast = lkw + n - 1;
                point();
            }
        }
    };
    {
        // the first segment is valid (k1 > k0); a wave without k-steps in it
        // still points at it (k-step k0) before looking further
        const int n = dec_items<NKQ>(ls, kq, &lkw);
        point();
        lrem = (n + kDecStages - 1) / kDecStages * kDecStages;
        lk = n > 0 ? lkw : ls.k0;
        llast = n > 0 ? lkw + n - 1 : ls.k0;
        if (lrem == 0) advance();
    }
    const unsigned lo16 = (unsigned)l * 16u, lo4 = (unsigned)l * 4u, lsc = (unsigned)(l & 15) * 2u;
    auto issue = [&](u32x4 (&xa)[MB], u32x4 (&wb)[NB]) __attribute__((always_inline)) {
        if (lrem == 0 && ls.valid) advance();
        const int kk = min(lk, llast);        // padding (and the end) repeats the last load
        if (ls.valid && lrem > 0) {
            ++lk;
            --lrem;
        }
        if (Q4 && lq) {
            const unsigned qo = (unsigned)kk * kInt4FragBytes + lo4, so = (unsigned)(kk / kInt4Group) * 32u + lsc;
#pragma unroll
            for (int c = 0; c < NB; ++c)
                wb[c] = u32x4{*reinterpret_cast<const uint32_t*>(wbp[c] + qo),
                              (uint32_t)*reinterpret_cast<const uint16_t*>(sbp[c] + so), 0u, 0u};
        } else {
            const unsigned fo = (unsigned)kk * 1024u + lo16;
#pragma unroll
            for (int c = 0; c < NB; ++c) wb[c] = *reinterpret_cast<const u32x4*>(wbp[c] + fo);
        }
        const unsigned xo = XR ? (unsigned)kk * 64u : (unsigned)kk * 1024u + lo16;
#pragma unroll
        for (int rb = 0; rb < MB; ++rb) xa[rb] = *reinterpret_cast<const u32x4*>(xb[rb] + xo);
    };

    u32x4 xs[kDecStages][MB], ws[kDecStages][NB];
#pragma unroll
    for (int d = 0; d < kDecStages; ++d) issue(xs[d], ws[d]);
    f32x4 acc[MB][NB];
#pragma unroll
    for (int rb = 0; rb < MB; ++rb)
#pragma unroll
        for (int cb = 0; cb < NB; ++cb) acc[rb][cb] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (;;) {
        int ckw;
        const int n = dec_items<NKQ>(cs, kq, &ckw);
        const bool cq = Q4 && a.p[cs.p].Ws && 4 * cs.gl < a.p[cs.p].nWb;   // INT4 base blocks
        for (int i = 0; i < n; i += kDecStages) {
#pragma unroll
            for (int d = 0; d < kDecStages; ++d) {
                if (i + d < n) {
                    if (Q4 && cq)
                        mma_nb_int4<MB, NB>(acc, xs[d], ws[d]);
                    else
                        mma_nb<MB, NB>(acc, xs[d], ws[d]);
                }
                issue(xs[d], ws[d]);
            }
        }
        dec_flush<MB, NB>(a, cs, acc, red, b);
        dec_next(a, n_act_v, gr, se, cs);
        if (!cs.valid) break;
    }
}

hipError_t launch_dec_main(const DecArgs& a, int mb, hipStream_t s) {
    const int grid = a.main_grid;
    if (grid <= 0 || grid > kDecMaxGrid) return hipErrorInvalidValue;
    bool q4 = false;
    for (int i = 0; i < a.n_proj; ++i) q4 = q4 || a.p[i].Ws != nullptr;
    if (a.plan) {
        // the planning form reads one or two row blocks of the caller's X
        if (mb != 1 && mb != 2) return hipErrorInvalidValue;
        for (int i = 0; i < a.n_proj; ++i)
            if (!a.p[i].X) return hipErrorInvalidValue;
        if (mb == 1 && q4)
            hipLaunchKernelGGL((dec_main_kernel<1, true, true>), dim3(grid), dim3(kDecThreads), 0, s, a);
        else if (mb == 1)
            hipLaunchKernelGGL((dec_main_kernel<1, false, true>), dim3(grid), dim3(kDecThreads), 0, s, a);
        else if (q4)
            hipLaunchKernelGGL((dec_main_kernel<2, true, true>), dim3(grid), dim3(kDecThreads), 0, s, a);
        else
            hipLaunchKernelGGL((dec_main_kernel<2, false, true>), dim3(grid), dim3(kDecThreads), 0, s, a);
        return hipGetLastError();
    }
#define BDL_DEC_CASE(M)                                                                                   \
    case M:                                                                                               \
        if (q4)                                                                                           \
            hipLaunchKernelGGL((dec_main_kernel<M, true, false>), dim3(grid), dim3(kDecThreads), 0, s, a);  \
        else                                                                                              \
            hipLaunchKernelGGL((dec_main_kernel<M, false, false>), dim3(grid), dim3(kDecThreads), 0, s, a); \
        break;
    switch (mb) {
        BDL_DEC_CASE(1)
        BDL_DEC_CASE(2)
        BDL_DEC_CASE(3)
        BDL_DEC_CASE(4)
        default: return hipErrorInvalidValue;
    }
#undef BDL_DEC_CASE
    return hipGetLastError();
}

// Workgroups of the main launch holding k-steps of group gl of projection pp:
// the owners of its first and of its last k-step (every one between owns at
// least one, since each workgroup's range spans at least one k-step).
__device__ __forceinline__ void group_wgs(const ProjPos& pp, int gl, unsigned U, int G, int* b0, int* b1) {
    const int wdt = min(4, pp.nb - 4 * gl);
    const unsigned goff = pp.ub + 4u * gl * pp.KS;
    *b0 = dec_wg_of(goff, U, G);
    *b1 = dec_wg_of(goff + (unsigned)(pp.KS - 1) * wdt, U, G);
}

constexpr int kEpiSeg = 8;     // partial tiles of an output group loaded in the first pass
constexpr int kEpiZSeg = 4;    // partial tiles of a Z group loaded in the first pass

__device__ __forceinline__ void add8(float (&acc)[8], const float4& a0, const float4& a1) {
    acc[0] += a0.x; acc[1] += a0.y; acc[2] += a0.z; acc[3] += a0.w;
    acc[4] += a1.x; acc[5] += a1.y; acc[6] += a1.z; acc[7] += a1.w;
}

__device__ __forceinline__ float4 ldf4(const float* p) { return *reinterpret_cast<const float4*>(p); }

// acc[c] += sc * sum_e z[e] * B^T[c][e] for the 8 ranks held in q[c]
__device__ __forceinline__ void expand8(float (&acc)[8], const float (&z)[8], const u32x4 (&q)[8], float sc) {
#pragma unroll
    for (int c = 0; c < 8; ++c) {
        const uint32_t qq[4] = {q[c].x, q[c].y, q[c].z, q[c].w};
        float sum = 0.f;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            sum = fmaf(z[2 * e], __uint_as_float(qq[e] << 16), sum);
            sum = fmaf(z[2 * e + 1], __uint_as_float(qq[e] & 0xffff0000u), sum);
        }
        acc[c] = fmaf(sc, sum, acc[c]);
    }
}

// The 8 outputs of token t in columns col .. col + 7 of output tile n of
// projection p: the tile's partials added in workgroup order, plus scale *
// sum_j Z[t, j] B^T[col + c, j] with Z from the partials of the token's own
// adapter, all in fp32.  Tokens of one adapter share their B^T lines inside a
// workgroup, so each tile reads each used adapter's B once.  After the
// token's id, rank and group are known, every load of the base partials, of
// the first 16 ranks' B^T and of their Z partials is issued before any sum,
// so a thread waits for two round trips (more only for ranks above 16 or
// groups split over many workgroups).
// bs: this thread's columns' ranks 0..15 of B^T for token t, staged in LDS by
// dec_epi_stage (column c of the thread at bs[16 c], rank halves at +0, +1).
__device__ __forceinline__ void epi_acc(const DecArgs& a, int p, int n, int t, int col, const u32x4* bs,
                                        float (&acc)[8]) {
    const DecProj& P = a.p[p];
    const int v = a.vid[t];
    const int r8s = a.tr8[t];
    const int ai = a.tgrp[t];
    const ProjPos pp = dec_pos(a, p);
    const unsigned U = a.units;
    const int G = a.main_grid;

    // base partials of this tile
    int b0, b1;
    group_wgs(pp, n, U, G, &b0, &b1);
    const float* ysrc = a.part + (size_t)(pp.gb + n + b0) * kPartElems + t * 64 + (col - n * 64);
    // loads are unconditional with the index clamped to the last slot, so the
    // compiler issues them all before the first sum
    float4 y[kEpiSeg][2];
#pragma unroll
    for (int j = 0; j < kEpiSeg; ++j) {
        const size_t o = (size_t)min(j, b1 - b0) * kPartElems;
        y[j][0] = ldf4(ysrc + o);
        y[j][1] = ldf4(ysrc + o + 4);
    }

    // LoRA operands of ranks 0..15: B^T rows and Z partials
    const bool lora = r8s > 0 && ai >= 0;
    int sig = 0;
#pragma unroll
    for (int q = 1; q < kMaxSlices; ++q)
        if (q < P.n_slices && col >= P.slice_col[q]) sig = q;
    const uint16_t* bb = a.pool + (size_t)max(v, 0) * a.slot_stride + P.b_off + (size_t)col * r8s;
    float sc = 0.f;
    u32x4 q[2][8];
    float4 zp[2][kEpiZSeg][2];
    int z0[2] = {0, 0}, z1[2] = {-1, -1};
    const float* zsrc[2] = {nullptr, nullptr};
    if (lora) {
        sc = a.scale[v];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            if (8 * h < r8s) {
#pragma unroll
                for (int c = 0; c < 8; ++c) q[h][c] = bs[16 * c + h];
                const int vc = sig * r8s + 8 * h;
                const int vb = P.nWb + ai * P.nbA + (vc >> 4);
                group_wgs(pp, vb >> 2, U, G, &z0[h], &z1[h]);
                zsrc[h] = a.part + (size_t)(pp.gb + (vb >> 2) + z0[h]) * kPartElems + t * 64 + (vb & 3) * 16 + (vc & 15);
#pragma unroll
                for (int j = 0; j < kEpiZSeg; ++j) {
                    const size_t o = (size_t)min(j, z1[h] - z0[h]) * kPartElems;
                    zp[h][j][0] = ldf4(zsrc[h] + o);
                    zp[h][j][1] = ldf4(zsrc[h] + o + 4);
                }
            }
        }
    }

#pragma unroll
    for (int c = 0; c < 8; ++c) acc[c] = 0.f;
#pragma unroll
    for (int j = 0; j < kEpiSeg; ++j)
        if (b0 + j <= b1) add8(acc, y[j][0], y[j][1]);
    for (int j0 = kEpiSeg; j0 <= b1 - b0; j0 += kEpiSeg) {
        float4 yy[kEpiSeg][2];
#pragma unroll
        for (int j = 0; j < kEpiSeg; ++j) {
            const size_t o = (size_t)min(j0 + j, b1 - b0) * kPartElems;
            yy[j][0] = ldf4(ysrc + o);
            yy[j][1] = ldf4(ysrc + o + 4);
        }
#pragma unroll
        for (int j = 0; j < kEpiSeg; ++j)
            if (j0 + j <= b1 - b0) add8(acc, yy[j][0], yy[j][1]);
    }
    if (lora) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            if (8 * h < r8s) {
                float z[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int j = 0; j < kEpiZSeg; ++j)
                    if (z0[h] + j <= z1[h]) add8(z, zp[h][j][0], zp[h][j][1]);
                for (int j0 = kEpiZSeg; j0 <= z1[h] - z0[h]; j0 += kEpiZSeg) {
                    float4 zz[kEpiZSeg][2];
#pragma unroll
                    for (int j = 0; j < kEpiZSeg; ++j) {
                        const size_t o = (size_t)min(j0 + j, z1[h] - z0[h]) * kPartElems;
                        zz[j][0] = ldf4(zsrc[h] + o);
                        zz[j][1] = ldf4(zsrc[h] + o + 4);
                    }
#pragma unroll
                    for (int j = 0; j < kEpiZSeg; ++j)
                        if (j0 + j <= z1[h] - z0[h]) add8(z, zz[j][0], zz[j][1]);
                }
                expand8(acc, z, q[h], sc);
            }
        }
        // ranks 16 and up, 8 at a time (two octets per turn, so that the
        // loads of both are in flight together)
#pragma unroll 2
        for (int j0 = 16; j0 < r8s; j0 += 8) {
            u32x4 qr[8];
#pragma unroll
            for (int c = 0; c < 8; ++c) qr[c] = ld16(bb + (size_t)c * r8s + j0);
            const int vc = sig * r8s + j0;
            const int vb = P.nWb + ai * P.nbA + (vc >> 4);
            int c0, c1;
            group_wgs(pp, vb >> 2, U, G, &c0, &c1);
            const float* src = a.part + (size_t)(pp.gb + (vb >> 2)) * kPartElems + t * 64 + (vb & 3) * 16 + (vc & 15);
            float z[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
            for (int j0 = 0; j0 <= c1 - c0; j0 += kEpiZSeg) {
                float4 zz[kEpiZSeg][2];
#pragma unroll
                for (int j = 0; j < kEpiZSeg; ++j) {
                    const float* s2 = src + (size_t)(c0 + min(j0 + j, c1 - c0)) * kPartElems;
                    zz[j][0] = ldf4(s2);
                    zz[j][1] = ldf4(s2 + 4);
                }
#pragma unroll
                for (int j = 0; j < kEpiZSeg; ++j)
                    if (j0 + j <= c1 - c0) add8(z, zz[j][0], zz[j][1]);
            }
            expand8(acc, z, qr, sc);
        }
    }
}

__device__ __forceinline__ u32x4 pack_bf16x8(const float (&v)[8]) {
    u32x4 o;
    o.x = (uint32_t)f2bf(v[0]) | ((uint32_t)f2bf(v[1]) << 16);
    o.y = (uint32_t)f2bf(v[2]) | ((uint32_t)f2bf(v[3]) << 16);
    o.z = (uint32_t)f2bf(v[4]) | ((uint32_t)f2bf(v[5]) << 16);
    o.w = (uint32_t)f2bf(v[6]) | ((uint32_t)f2bf(v[7]) << 16);
    return o;
}

// One workgroup per 64-column output tile, all tokens: thread (t, g) computes
// the 8 outputs of token t in columns 8 g .. 8 g + 7 of the tile.  In MLP mode
// the tiles are those of projection 0 only, and the outputs become the MLP
// intermediate H = out_0 (act none) or silu(out_0) * out_1 (act silu_mul,
// projection 1 being up), stored in bf16 in the fragment layout the second
// projection reads (rows = tokens, k = these columns).
// Epilogue workgroups: kEpiTok tokens x 8 column octets of one 64-column tile.
constexpr int kEpiTok = 8;
constexpr int kEpiThreads = kEpiTok * 8;

// Ranks 0..15 of B^T for the workgroup's tokens and 64-column tile n of
// projection p, into LDS: 16-byte pieces in which consecutive threads read
// consecutive (column, rank half) pieces of a token's slice, so a wave's load
// covers contiguous bytes (a thread loading its own 8 columns would touch a
// cache line per lane).  A token's slice is stored column-interleaved: column
// c in slot (c mod 8) 8 + c / 8, 32 bytes, so the 8 threads of a token reading
// their k-th column read consecutive slots.  Pieces past the rank or the
// projection's width read a valid piece, unused.  Starts and ends with a
// barrier (every thread of the workgroup calls it).
__device__ __forceinline__ void dec_epi_stage(const DecArgs& a, int p, int n, int t, u32x4* bst, int2* rinf) {
    const DecProj& P = a.p[p];
    if ((threadIdx.x & 7) == 0) {
        const int v = a.vid[t];
        rinf[threadIdx.x >> 3] = make_int2(max(v, 0), v >= 0 ? min(a.tr8[t], kMaxRank8) : 0);
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kEpiTok * 128 / kEpiThreads; ++k) {
        const int idx = k * kEpiThreads + threadIdx.x, row = idx >> 7, pc = idx & 127, c = pc >> 1, h = pc & 1;
        const int2 inf = rinf[row];
        const int colc = min(n * 64 + c, P.N - 1), hh = 8 * h < inf.y ? 8 * h : 0;
        bst[(row * 64 + (c & 7) * 8 + (c >> 3)) * 2 + h] =
            ld16(a.pool + (size_t)inf.x * a.slot_stride + P.b_off + (size_t)colc * inf.y + hh);
    }
    __syncthreads();
}

// SILU: the MLP's gated mode (gate and up summed, H = silu(gate) * up).
template <bool SILU>
__global__ __launch_bounds__(kEpiThreads) void dec_epi_kernel(DecArgs a) {
    const int tile = blockIdx.x;
    int p = 0;
#pragma unroll
    for (int q = 1; q < kMaxProjs; ++q)
        if (q < a.n_proj && tile >= a.stb[q]) p = q;
    const DecProj& P = a.p[p];
    const int n = tile - a.stb[p];
    const int t = blockIdx.y * kEpiTok + (threadIdx.x >> 3);
    const int col = n * 64 + (threadIdx.x & 7) * 8;
    // threads past the last token or column compute on clamped indices and
    // store nothing (no early exit: every load is issued without waiting on
    // a branch)
    const bool live = t < a.T && col < P.N;
    const int tt = min(t, a.T - 1), cc = min(col, P.N - 8);
    __shared__ u32x4 bst[kEpiTok * 64 * 2];
    __shared__ int2 rinf[kEpiTok];
    const u32x4* bs = bst + ((threadIdx.x >> 3) * 64 + (cc - n * 64) / 8) * 2;
    float acc[8];
    dec_epi_stage(a, p, n, tt, bst, rinf);
    epi_acc(a, p, n, tt, cc, bs, acc);
    if constexpr (SILU) {
        // every thread stages and sums up as well (the barriers are uniform)
        float up[8];
        dec_epi_stage(a, 1, n, tt, bst, rinf);
        epi_acc(a, 1, n, tt, cc, bs, up);
#pragma unroll
        for (int c = 0; c < 8; ++c) acc[c] = acc[c] / (1.f + __expf(-acc[c])) * up[c];
    }
    if (!live) return;
    if (a.mlp_act < 0) {
        *reinterpret_cast<u32x4*>(P.out + (size_t)t * P.N + col) = pack_bf16x8(acc);
        return;
    }
    // H[t][col .. col + 7] -> fragment (t / 16, col / 32), lane (t % 16) + 16 ((col % 32) / 8)
    const size_t f = ((size_t)(t >> 4) * a.h_KS + (col >> 5)) * kFrag + ((t & 15) + 16 * ((col & 31) >> 3)) * 8;
    *reinterpret_cast<u32x4*>(a.h_dst + f) = pack_bf16x8(acc);
}

hipError_t launch_dec_epi(const DecArgs& a, hipStream_t s) {
    const int grid = a.mlp_act < 0 ? a.tiles : (a.p[0].N + 63) / 64;
    if (grid <= 0) return hipSuccess;
    if (a.T > kDecodeMaxT || a.main_grid <= 0) return hipErrorInvalidValue;
    if (a.mlp_act >= 0 && (!a.h_dst || (a.mlp_act == BDLORA_ACT_SILU_MUL && (a.n_proj != 2 || a.p[1].N != a.p[0].N))))
        return hipErrorInvalidValue;
    const dim3 g(grid, (a.T + kEpiTok - 1) / kEpiTok);
    if (a.mlp_act == BDLORA_ACT_SILU_MUL)
        hipLaunchKernelGGL(dec_epi_kernel<true>, g, dim3(kEpiThreads), 0, s, a);
    else
        hipLaunchKernelGGL(dec_epi_kernel<false>, g, dim3(kEpiThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace bdl
