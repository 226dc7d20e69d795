// Prep launch of a forward call: workgroup 0 plans the batch, the others pack
// the activations into the MFMA fragment layout.  Decode batches take a
// one-wave plan that writes only what the decode launches read.
//
// Plan outputs (integer work, compared bit-exactly with the host plan):
//   vid[t]      validated id (-1: none or invalid; invalid ones raise *err)
//   tr8[t]      rank (padded to 8) of token t's adapter, 0 if none
//   tgrp[t]     (when asked for) group index of token t's adapter, -1 if none
//   groups      (slot, start, count) per adapter in use, slots ascending
//   perm        tokens group after group, ascending inside a group
//   items       shrink work items {slot, first perm index, rows <= mts, r8}
//   tile_oct    (when asked for) per base-GEMM row tile: the 8-rank octets of
//               every adapter present in the tile, slots ascending, code =
//               slot<<12 | r8<<4 | octet, followed by kOctTail entries of -1
//               (fewer at the end of the tile's oct_cap entries)
// Tokens are grouped by adapter (a counting sort over slots) so that every
// adapter's factors are streamed once per batch (heterogeneous batching of
// unmerged adapters, paper Sec. 1 and Sec. 2).
#include "bdl_device.h"

namespace bdl {

constexpr int kOctTail = 36;   // -1 entries after an octet list's last code (see the octet lists below)

// inclusive prefix sum over the 64 lanes of a wave (DPP row shifts, then row
// broadcasts of lanes 15 and 31)
__device__ __forceinline__ int wave_incl_scan(int v) {
    v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xf, 0xf, false);   // row_shr:1
    v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xf, 0xf, false);   // row_shr:2
    v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xf, 0xf, false);   // row_shr:4
    v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xf, 0xf, false);   // row_shr:8
    v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xa, 0xf, false);   // row_bcast:15
    v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xc, 0xf, false);   // row_bcast:31
    return v;
}

__device__ __forceinline__ int wave_total(int incl) { return __builtin_amdgcn_readlane(incl, 63); }


// Segments form: lane i < n_seg writes the id of segment i into ids_lds for
// its tokens (the host checked that the segments tile 0..T-1), and lane t
// reads token t's id back.
__device__ __forceinline__ int decode_seg_id(const PrepArgs& a, int* ids_lds) {
    const int l = threadIdx.x & 63;
    if (l < a.n_seg) {
        const int s0 = a.seg_start[l], s1 = l + 1 < a.n_seg ? a.seg_start[l + 1] : a.T, v = a.seg_slot[l];
        for (int t = s0; t < s1 && t < kDecodeMaxT; ++t) ids_lds[t] = v;
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);        // lgkmcnt(0): this wave's LDS stores are done
    __builtin_amdgcn_wave_barrier();
    return l < a.T ? ids_lds[l] : -1;
}

// Plan of a decode batch (T <= 64) by one wave: validated ids, ranks, the
// adapters in use in ascending slot order (groups) and each token's group.
// Lane t holds token t.  Pools of at most 64 slots keep the slot tables in
// lanes (one load round trip) and find the groups from the bit mask of slots
// in use; larger pools look the tables up per token and take the smallest
// remaining slot per pass.
__device__ void decode_plan(const PrepArgs& a, int* ids_lds) {
    const int l = threadIdx.x & 63;
    const bool in = l < a.T;
    const bool small = a.max_slots <= 64;
    const int lt = small && l < a.max_slots ? a.loaded[l] : 0;
    const int rt = small && l < a.max_slots ? a.r8[l] : 0;
    const int id = a.ids ? (in ? a.ids[l] : -1) : decode_seg_id(a, ids_lds);
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
    int g = 0, mine = -1;
    const int v = ok ? id : -1;
    if (small) {
        const unsigned long long bit = ok ? 1ull << v : 0ull;
        const unsigned long long used =
            (unsigned long long)wave_or((unsigned)bit) | ((unsigned long long)wave_or((unsigned)(bit >> 32)) << 32);
        const unsigned long long below = (1ull << l) - 1ull;
        if ((used >> l) & 1ull) {
            a.gslot[__popcll(used & below)] = l;
            if (a.gr8) a.gr8[__popcll(used & below)] = rt;   // lane l holds slot l's rank
        }
        if (ok) mine = __popcll(used & (bit - 1ull));
        g = __popcll(used);
    } else {
        unsigned long long rem = __ballot(ok);
        while (rem) {
            const int m = wave_min(((rem >> l) & 1ull) ? v : 0x7fffffff);
            const bool eq = ok && v == m;
            if (eq) mine = g;
            // slot m's rank: held by every lane whose token uses it
            const int rm = __builtin_amdgcn_readlane(r8v, __ffsll((long long)__ballot(eq)) - 1);
            if (l == 0) {
                a.gslot[g] = m;
                if (a.gr8) a.gr8[g] = rm;
            }
            ++g;
            rem &= ~__ballot(eq);
        }
    }
    // adapters past the launches' bound (possible only when a captured
    // forward replays after more adapters were loaded): base only, flagged
    if (a.act_max >= 0 && g > a.act_max) {
        const bool over = ok && mine >= a.act_max;
        bad = bad || __ballot(over) != 0ull;
        if (over) {
            ok = false;
            mine = -1;
        }
        g = a.act_max;
    }
    if (in) {
        a.vid[l] = ok ? v : -1;
        a.tr8[l] = ok ? r8v : 0;
        if (a.tgrp) a.tgrp[l] = mine;
    }
    if (l == 0) {
        a.meta[0] = g;
        a.meta[1] = 0;
        if (bad) atomicOr(a.err, 1);
    }
}

// activations -> fragment layout (all workgroups but 0)
// Each wave packs PER consecutive fragments per turn (consecutive k-steps of
// a row block, so a row's PER x 64 bytes are contiguous), all loads before
// the stores.  Batches from a few thousand fragments up take 4 (fewer,
// longer streams, each row's 256 bytes in whole lines: 70B layer at 256
// tokens, 15.5 -> 14.2 us); decode batches 1 (more waves issue their single
// load at once).
constexpr int kPackWide = 4;
constexpr int kPackWideFrags = 4096;    // total fragments from which the wide form is used

template <int PER>
__device__ void pack_activations(const PrepArgs& a, int blk, int nblk) {
    const int l = threadIdx.x & 63;
    for (int f0 = (blk * 16 + (threadIdx.x >> 6)) * PER; f0 < a.total_frags; f0 += nblk * 16 * PER) {
        u32x4 v[PER];
        uint16_t* dst[PER];
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int f = min(f0 + i, a.total_frags - 1);
            int j = 0;
            while (j + 1 < a.n_jobs && f >= a.jobs[j + 1].frag_base) ++j;
            const PackJob& J = a.jobs[j];
            const int KS = J.K >> 5;
            const int local = f - J.frag_base;
            const int rb = local / KS, ks = local - rb * KS;
            const int row = rb * 16 + (l & 15);
            v[i] = row < J.rows ? ld16(J.src + (size_t)row * J.K + ks * 32 + (l >> 4) * 8) : u32x4{0u, 0u, 0u, 0u};
            dst[i] = J.dst + (size_t)local * kFrag + l * 8;
        }
#pragma unroll
        for (int i = 0; i < PER; ++i)
            if (f0 + i < a.total_frags) *reinterpret_cast<u32x4*>(dst[i]) = v[i];
    }
}

// Stable placement by all 16 waves (batches of more than 1024 tokens, at
// most kPlanWaveGroups adapters, pools of at most kPlanParMaxSlots slots,
// ids in LDS; smaller batches count each token's rank directly): wave w
// takes the tokens [w C, (w + 1) C) and counts them per group into its LDS
// row wh[w][g]; a prefix over the waves turns the counts into each wave's
// first position per group (and for the tokens without an adapter); then
// every wave places its tokens chunk by chunk in token order.  A 64-token
// chunk of one adapter (prefill requests) is placed by one ballot; in a
// chunk of several, each lane counts the lanes before it in its group from
// the chunk's group ids staged in LDS (cgw), reads its group's position from
// the wave's row, and the group's last lane moves it on.  The positions
// equal those of the serial placement (stable in token order).
__device__ void place_waves(const PrepArgs& a, const int* vid_l, const int* ldl, const int* r8l, int* wh,
                            int* cg_l, const int* gstart_l, int* wnone, int n_groups, int n_ad) {
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const unsigned long long lt = (1ull << lane) - 1ull;
    const int C = (a.T + 16 * 64 - 1) / (16 * 64) * 64;
    const int t0 = min(wv * C, a.T), t1 = min(t0 + C, a.T);
    int* row = wh + wv * kPlanWaveGroups;
    int* cgw = cg_l + wv * 64;
    for (int g = lane; g < n_groups; g += 64) row[g] = 0;
    int nn = 0;
    for (int base = t0; base < t1; base += 64) {
        const int t = base + lane;
        const int v = t < t1 ? vid_l[t] : -2;
        const int g = v >= 0 ? ldl[v] : -1;
        const unsigned long long act = __ballot(v >= 0);
        if (act) {
            const int gl = __builtin_amdgcn_readlane(g, __ffsll((long long)act) - 1);
            const unsigned long long m = __ballot(v >= 0 && g == gl);
            if (m == act) {
                if (lane == 0) row[gl] += __popcll(m);
            } else if (v >= 0) {
                atomicAdd(&row[g], 1);
            }
        }
        nn += __popcll(__ballot(v == -1));
    }
    if (lane == 0) wnone[wv] = nn;
    __syncthreads();
    for (int g = tid; g < n_groups; g += 1024) {
        int r = gstart_l[g];
        for (int w = 0; w < 16; ++w) {
            const int c = wh[w * kPlanWaveGroups + g];
            wh[w * kPlanWaveGroups + g] = r;
            r += c;
        }
    }
    if (tid == 0) {
        int r = n_ad;
        for (int w = 0; w < 16; ++w) {
            const int c = wnone[w];
            wnone[w] = r;
            r += c;
        }
    }
    __syncthreads();
    int noff = wnone[wv];
    for (int base = t0; base < t1; base += 64) {
        const int t = base + lane;
        const int v = t < t1 ? vid_l[t] : -2;
        const int g = v >= 0 ? ldl[v] : -1;
        const unsigned long long act = __ballot(v >= 0);
        if (act) {
            const int gl = __builtin_amdgcn_readlane(g, __ffsll((long long)act) - 1);
            const unsigned long long m = __ballot(v >= 0 && g == gl);
            if (m == act) {
                // one group: its position from the row (one uniform read)
                const int b0 = row[gl];
                if (v >= 0) {
                    const int pos = b0 + __popcll(m & lt);
                    a.perm[pos] = t;
                    if (a.rowtok) a.rowtok[pos] = t;
                    if (a.rowslot) a.rowslot[pos] = (r8l[v] << 16) | v;
                }
                if (lane == 0) row[gl] = b0 + __popcll(m);
            } else {
                cgw[lane] = g;                        // (in order with the reads below)
                int before = 0;
                bool later = false;
#pragma unroll 4
                for (int j = 0; j < 64; j += 4) {
                    const int4 q = *reinterpret_cast<const int4*>(cgw + j);
                    before += (j < lane && q.x == g) + (j + 1 < lane && q.y == g) + (j + 2 < lane && q.z == g) +
                              (j + 3 < lane && q.w == g);
                    later = later || (j > lane && q.x == g) || (j + 1 > lane && q.y == g) ||
                            (j + 2 > lane && q.z == g) || (j + 3 > lane && q.w == g);
                }
                if (v >= 0) {
                    const int pos = row[g] + before;
                    a.perm[pos] = t;
                    if (a.rowtok) a.rowtok[pos] = t;
                    if (a.rowslot) a.rowslot[pos] = (r8l[v] << 16) | v;
                    if (!later) row[g] = pos + 1;     // the group's last lane in the chunk
                }
            }
        }
        const unsigned long long um = __ballot(v == -1);
        if (v == -1 && a.rowtok) {
            const int pos = noff + __popcll(um & lt);
            a.rowtok[pos] = t;
            if (a.rowslot) a.rowslot[pos] = -1;
        }
        noff += __popcll(um);
    }
}

__global__ __launch_bounds__(1024) void prep_kernel(PrepArgs a) {
    if (blockIdx.x > 0) {
        if (a.total_frags >= kPackWideFrags)
            pack_activations<kPackWide>(a, blockIdx.x - 1, gridDim.x - 1);
        else
            pack_activations<1>(a, blockIdx.x - 1, gridDim.x - 1);
        return;
    }
    __shared__ int vid_l[kPlanLdsTokens];
    if (a.decode_plan) {
        if (threadIdx.x < 64) decode_plan(a, vid_l);
        return;
    }
    extern __shared__ int tabs[];             // cnt | r8 | loaded | 15 tile bitmaps
    const int nwords = (a.max_slots + 31) >> 5;
    int* cnt = tabs;                          // counts, then group starts
    int* r8l = tabs + a.max_slots;
    int* ldl = tabs + 2 * a.max_slots;
    unsigned* bits = reinterpret_cast<unsigned*>(tabs + 3 * a.max_slots);
    __shared__ int s_err;
    __shared__ int seg_s[kMaxSeg], seg_v[kMaxSeg];
    __shared__ int wsum[16][3];
    __shared__ int wpre[16][3];
    __shared__ int gstart_l[kPlanWaveGroups];   // group tables (the first kPlanWaveGroups groups):
    __shared__ int gcount_l[kPlanWaveGroups];   // start, count and slot, read by the
    __shared__ int gslot_l[kPlanWaveGroups];    // placement and the octet lists
    __shared__ int wnone[16];
    __shared__ __align__(16) int cg_l[16 * 64];   // place_waves: a chunk's group ids, per wave
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const bool in_lds = a.T <= kPlanLdsTokens;

    for (int s = tid; s < a.max_slots; s += 1024) {
        cnt[s] = 0;
        r8l[s] = a.r8[s];
        ldl[s] = a.loaded[s];
    }
    if (tid == 0) s_err = 0;
    if (!a.ids && tid < a.n_seg) {
        seg_s[tid] = a.seg_start[tid];
        seg_v[tid] = a.seg_slot[tid];
    }
    __syncthreads();
    // id of token t from the segments: the last segment starting at or
    // before t (binary search; seg_s[0] = 0)
    auto seg_id = [&](int t) {
        int lo = 0, hi = a.n_seg - 1;
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (seg_s[mid] <= t)
                lo = mid;
            else
                hi = mid - 1;
        }
        return seg_v[lo];
    };
    // ids in batches of 8 per thread: all loads of a batch are issued before
    // any of its stores, so a batch costs one round trip
    for (int t0 = 0; t0 < a.T; t0 += 8 * 1024) {
        int idv[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int t = t0 + j * 1024 + tid;
            idv[j] = t < a.T ? (a.ids ? a.ids[t] : seg_id(t)) : -1;
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            if (t0 + j * 1024 + (tid & ~63) >= a.T) break;   // the wave's tokens are all past T
            const int t = t0 + j * 1024 + tid;
            const int id = idv[j];
            const bool ok = t < a.T && id >= 0 && id < a.max_slots && ldl[id] != 0;
            if (t < a.T) {
                if (!ok && id != -1) s_err = 1;
                const int v = ok ? id : -1;
                a.vid[t] = v;
                a.tr8[t] = ok ? r8l[id] : 0;
                if (in_lds) vid_l[t] = v;
            }
            // a wave whose tokens share one adapter (a prefill request) adds
            // its count once; others add per token
            const unsigned long long act = __ballot(ok);
            if (act) {
                const int il = __builtin_amdgcn_readlane(id, __ffsll((long long)act) - 1);
                const unsigned long long m = __ballot(ok && id == il);
                if (m == act) {
                    if (lane == 0) atomicAdd(&cnt[il], __popcll(m));
                } else if (ok) {
                    atomicAdd(&cnt[id], 1);
                }
            }
        }
    }
    __syncthreads();

    // exclusive scan over slots of (tokens, groups, shrink items)
    const int per = (a.max_slots + 1023) / 1024;
    const int s0 = min(tid * per, a.max_slots), s1 = min(s0 + per, a.max_slots);
    int tok = 0, grp = 0, itm = 0;
    for (int s = s0; s < s1; ++s) {
        const int c = cnt[s];
        tok += c;
        grp += c > 0;
        itm += (c + a.mts - 1) / a.mts;
    }
    const int it = wave_incl_scan(tok), ig = wave_incl_scan(grp), ii = wave_incl_scan(itm);
    if (lane == 63) {
        wsum[wv][0] = it;
        wsum[wv][1] = ig;
        wsum[wv][2] = ii;
    }
    __syncthreads();
    if (tid < 3) {
        int acc = 0;
        for (int w = 0; w < 16; ++w) {
            wpre[w][tid] = acc;
            acc += wsum[w][tid];
        }
    }
    __syncthreads();
    int tok_off = wpre[wv][0] + it - tok;
    int g_off = wpre[wv][1] + ig - grp;
    int i_off = wpre[wv][2] + ii - itm;
    for (int s = s0; s < s1; ++s) {
        const int c = cnt[s];
        if (c > 0) {
            ldl[s] = g_off;                   // group index of the slot (validation is done)
            if (g_off < kPlanWaveGroups) {
                gstart_l[g_off] = tok_off;
                gcount_l[g_off] = c;
                gslot_l[g_off] = s;
            }
            a.gslot[g_off] = s;
            a.gstart[g_off] = tok_off;
            a.gcount[g_off] = c;
            for (int r = 0; r < c; r += a.mts)
                a.items[i_off++] = make_int4(s, tok_off + r, min(a.mts, c - r), r8l[s]);
            ++g_off;
        }
        cnt[s] = tok_off;                     // group start for the placement below
        tok_off += c;
    }
    if (tid == 1023) {
        a.meta[0] = g_off;
        a.meta[1] = i_off;
        a.meta[2] = 0;
    }
    __syncthreads();
    if (a.tgrp)
        for (int t = tid; t < a.T; t += 1024) {
            const int v = in_lds ? vid_l[t] : a.vid[t];
            a.tgrp[t] = v >= 0 ? ldl[v] : -1;
        }

    // stable placement: perm[start(v) + #{t' < t : vid[t'] == v}] = t; with
    // rowtok, the same order followed by the tokens without an adapter
    // (rowtok[n_ad + #{t' < t : no adapter}] = t), a permutation of all rows
    const int n_ad = wpre[15][0] + wsum[15][0];   // tokens with an adapter
    const int n_groups_all = wpre[15][1] + wsum[15][1];
    if (a.T > 1024 && in_lds && n_groups_all <= kPlanWaveGroups && a.max_slots <= kPlanParMaxSlots) {
        place_waves(a, vid_l, ldl, r8l, tabs + 3 * a.max_slots + 15 * nwords, cg_l, gstart_l, wnone, n_groups_all,
                    n_ad);
    } else if (a.T <= 1024) {
        const int t = tid;
        const int v = t < a.T ? vid_l[t] : -1;
        if (v >= 0) {
            int rank = 0;
            for (int u = 0; u < t; ++u) rank += vid_l[u] == v;
            a.perm[cnt[v] + rank] = t;
            if (a.rowtok) a.rowtok[cnt[v] + rank] = t;
            if (a.rowslot) a.rowslot[cnt[v] + rank] = (r8l[v] << 16) | v;
        } else if (t < a.T && a.rowtok) {
            int rank = 0;
            for (int u = 0; u < t; ++u) rank += vid_l[u] < 0;
            a.rowtok[n_ad + rank] = t;
            if (a.rowslot) a.rowslot[n_ad + rank] = -1;
        }
    } else if (wv == 0) {
        int ubase = n_ad;
        for (int base = 0; base < a.T; base += 64) {
            const int t = base + lane;
            const int v = t < a.T ? (in_lds ? vid_l[t] : a.vid[t]) : -1;
            bool ok = v >= 0;
            const unsigned long long um = __ballot(t < a.T && !ok);
            if (a.rowtok && t < a.T && !ok) a.rowtok[ubase + __popcll(um & ((1ull << lane) - 1ull))] = t;
            if (a.rowslot && t < a.T && !ok) a.rowslot[ubase + __popcll(um & ((1ull << lane) - 1ull))] = -1;
            ubase += __popcll(um);
            unsigned long long act = __ballot(ok);
            while (act) {
                const int leader = __ffsll((long long)act) - 1;
                const int s = __shfl(v, leader);
                const bool mine = ok && v == s;
                const unsigned long long m = __ballot(mine);
                const int b = cnt[s];
                if (lane == leader) cnt[s] = b + __popcll(m);
                if (mine) {
                    const int pos = b + __popcll(m & ((1ull << lane) - 1ull));
                    a.perm[pos] = t;
                    if (a.rowtok) a.rowtok[pos] = t;
                    if (a.rowslot) a.rowslot[pos] = (r8l[s] << 16) | s;
                    ok = false;
                }
                act &= ~m;
            }
        }
    }

    // expand octet lists of the base-GEMM row tiles, one tile per wave.  A
    // list ends with kOctTail entries of -1: its readers take the codes in
    // groups of 4, the 64-row kernel's 8 waves a group each, 32 entries
    // apart, and stop at their first group of -1 (so they read at most 35
    // entries past the last code); the large tiles read the groups in order,
    // one group ahead.
    if (a.tile_oct && wv > 0) {
        const int mt = a.gemm_mt;
        const int tiles = (a.T + mt - 1) / mt;
        unsigned* bm = bits + (size_t)(wv - 1) * nwords;
        const int n_groups = wpre[15][1] + wsum[15][1];
        for (int m = wv - 1; m < tiles; m += 15) {
            int* dst = a.tile_oct + (size_t)m * a.oct_cap;
            if (a.oct_perm) {
                // rowtok order: block m holds rows [m mt, m mt + mt) of the
                // groups laid end to end (slot order, then the tokens without
                // an adapter): its adapters are the groups overlapping it,
                // read from the group tables (no need to wait for the
                // placement)
                const int r0 = m * mt, r1 = min(r0 + mt, n_ad);
                const bool gl = n_groups <= kPlanWaveGroups;   // tables in LDS
                int base = 0;
                for (int g0 = 0; g0 < n_groups; g0 += 64) {
                    const int g = g0 + lane;
                    const int gs = g < n_groups ? (gl ? gstart_l[g] : a.gstart[g]) : 0;
                    const int gc = g < n_groups ? (gl ? gcount_l[g] : a.gcount[g]) : 0;
                    const bool in = g < n_groups && gs < r1 && gs + gc > r0;
                    const int slot = in ? (gl ? gslot_l[g] : a.gslot[g]) : 0;
                    const int r8s = in ? r8l[slot] : 0;
                    const int c = r8s >> 3;
                    const int inc = wave_incl_scan(c);
                    int o = base + inc - c;
                    for (int j = 0; j < c; ++j) dst[o++] = (slot << 12) | (r8s << 4) | j;
                    base += wave_total(inc);
                }
                for (int i = base + lane; i < min(a.oct_cap, base + kOctTail); i += 64) dst[i] = -1;
                continue;
            }
            for (int i = lane; i < nwords; i += 64) bm[i] = 0u;
            __builtin_amdgcn_wave_barrier();
            const int t = m * mt + lane;
            const int v = (lane < mt && t < a.T) ? (in_lds ? vid_l[t] : a.vid[t]) : -1;
            if (v >= 0) atomicOr(&bm[v >> 5], 1u << (v & 31));
            __builtin_amdgcn_wave_barrier();
            int base = 0;
            for (int wb = 0; wb < nwords; wb += 64) {
                const int wi = wb + lane;
                const unsigned word = wi < nwords ? bm[wi] : 0u;
                int c = 0;
                for (unsigned b = word; b; b &= b - 1u) c += r8l[wi * 32 + __ffs(b) - 1] >> 3;
                const int inc = wave_incl_scan(c);
                int o = base + inc - c;
                for (unsigned b = word; b; b &= b - 1u) {
                    const int slot = wi * 32 + __ffs(b) - 1;
                    const int r8s = r8l[slot];
                    for (int j = 0; j < (r8s >> 3); ++j) dst[o++] = (slot << 12) | (r8s << 4) | j;
                }
                base += wave_total(inc);
            }
            for (int i = base + lane; i < min(a.oct_cap, base + kOctTail); i += 64) dst[i] = -1;
        }
    }
    if (tid == 0 && s_err) atomicOr(a.err, 1);
}

hipError_t launch_prep(const PrepArgs& a, hipStream_t s) {
    const int per = a.total_frags >= kPackWideFrags ? kPackWide : 1;
    int pack_blocks = (a.total_frags + 16 * per - 1) / (16 * per);
    if (pack_blocks > 4096) pack_blocks = 4096;
    const int nwords = (a.max_slots + 31) >> 5;
    size_t lds = a.decode_plan ? 0 : 3 * (size_t)a.max_slots * sizeof(int) + 15 * (size_t)nwords * sizeof(unsigned);
    // place_waves' per-wave counts, for the batches that take it
    if (!a.decode_plan && a.T > 1024 && a.max_slots <= kPlanParMaxSlots) lds += 16 * kPlanWaveGroups * sizeof(int);
    hipLaunchKernelGGL(prep_kernel, dim3(1 + pack_blocks), dim3(1024), lds, s, a);
    return hipGetLastError();
}

// MLP intermediate of a batch above the decode size: H = G (U null) or
// silu(G) * U from the first projections' fp32 outputs [T x N], rounded to
// bf16 and stored in the fragment layout of the second projection's input
// (rows padded to 16 with zeros).  Thread = 8 columns of one row.
__global__ __launch_bounds__(256) void mlp_pack_kernel(const float* G, const float* U, uint16_t* dst, int T, int N) {
    const int per_row = N >> 3;
    const long long u = (long long)blockIdx.x * 256 + threadIdx.x;
    const int rows = (T + 15) & ~15;
    if (u >= (long long)rows * per_row) return;
    const int row = (int)(u / per_row), col = (int)(u - (long long)row * per_row) * 8;
    u32x4 o = u32x4{0u, 0u, 0u, 0u};
    if (row < T) {
        const float4 g0 = *reinterpret_cast<const float4*>(G + (size_t)row * N + col);
        const float4 g1 = *reinterpret_cast<const float4*>(G + (size_t)row * N + col + 4);
        float h[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
        if (U) {
            const float4 u0 = *reinterpret_cast<const float4*>(U + (size_t)row * N + col);
            const float4 u1 = *reinterpret_cast<const float4*>(U + (size_t)row * N + col + 4);
            const float uv[8] = {u0.x, u0.y, u0.z, u0.w, u1.x, u1.y, u1.z, u1.w};
#pragma unroll
            for (int e = 0; e < 8; ++e) h[e] = h[e] / (1.f + __expf(-h[e])) * uv[e];
        }
        o.x = (uint32_t)f2bf(h[0]) | ((uint32_t)f2bf(h[1]) << 16);
        o.y = (uint32_t)f2bf(h[2]) | ((uint32_t)f2bf(h[3]) << 16);
        o.z = (uint32_t)f2bf(h[4]) | ((uint32_t)f2bf(h[5]) << 16);
        o.w = (uint32_t)f2bf(h[6]) | ((uint32_t)f2bf(h[7]) << 16);
    }
    const size_t f = ((size_t)(row >> 4) * (N >> 5) + (col >> 5)) * kFrag + ((row & 15) + 16 * ((col & 31) >> 3)) * 8;
    *reinterpret_cast<u32x4*>(dst + f) = o;
}

hipError_t launch_mlp_pack(const float* G, const float* U, uint16_t* dst, int T, int N, hipStream_t s) {
    if (T <= 0) return hipSuccess;
    if (N % 32) return hipErrorInvalidValue;
    const long long units = (long long)((T + 15) & ~15) * (N >> 3);
    hipLaunchKernelGGL(mlp_pack_kernel, dim3((unsigned)((units + 255) / 256)), dim3(256), 0, s, G, U, dst, T, N);
    return hipGetLastError();
}

}  // namespace bdl
