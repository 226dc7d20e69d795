// HIP kernels of the BD-LoRA shard forward for gfx950 (MI355X).
//
// A forward launch of one token batch over P projections (all sharing the
// tokens' adapter ids) runs three kernels on the caller's stream:
//
//  1. plan_kernel   -- validates ids and groups tokens by adapter (counting
//                      sort over slots, one workgroup).  Integer work only.
//  2. shrink_kernel -- Z = scale * X A for every adapter group (the LoRA
//                      "shrink", matmul_3 / matmul_5 of the paper's Fig. 2/3,
//                      line "Z <- X A" of Alg. 1 and Alg. 2).  Each group's
//                      factor A^T is streamed once; the group's token rows are
//                      gathered.
//  3. gemm_kernel   -- out = X W_s^T + Z B for each output tile: the base
//                      product (matmul_1 / matmul_2) with the LoRA "expand"
//                      (matmul_4 / matmul_6) and the add (add_1 / add_2)
//                      fused, one bf16 store per output (Alg. 1 / Alg. 2,
//                      lines "Y_adapter <- Z B" and "Y <- Y + Y_adapter").
//
// Both GEMM-shaped kernels use 8 waves per workgroup that split the K loop
// and reduce through LDS in a fixed order, so results are bitwise
// reproducible.  The expand runs as extra MFMA k-steps: for the adapters
// present in the tile, 8-rank pieces ("octets") of B^T are the B operand
// and the matching Z entries (zero for tokens of other adapters) the A
// operand.  Z is kept as a pair of bf16 numbers (hi + lo, about 16
// significant bits) and multiplied in two MFMAs, so the intermediate adds
// no bf16-sized error to the LoRA term.
#include "bdl_device.h"

namespace bdl {

// --------------------------------------------------------------------------
// 1. plan
// --------------------------------------------------------------------------

__global__ __launch_bounds__(1024) void plan_kernel(PlanArgs a) {
    extern __shared__ int cnt[];              // [max_slots]: counts, then cursors
    __shared__ int s_err;
    __shared__ int wsum[16][3];
    __shared__ int wpre[16][3];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;

    for (int s = tid; s < a.max_slots; s += 1024) cnt[s] = 0;
    if (tid == 0) s_err = 0;
    __syncthreads();
    for (int t = tid; t < a.T; t += 1024) {
        const int id = a.ids[t];
        const bool ok = id >= 0 && id < a.max_slots && a.loaded[id] != 0;
        if (!ok && id != -1) s_err = 1;
        a.vid[t] = ok ? id : -1;
        if (ok) atomicAdd(&cnt[id], 1);
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
    int it = tok, ig = grp, ii = itm;
    for (int d = 1; d < 64; d <<= 1) {
        const int t2 = __shfl_up(it, d), g2 = __shfl_up(ig, d), i2 = __shfl_up(ii, d);
        if (lane >= d) {
            it += t2;
            ig += g2;
            ii += i2;
        }
    }
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
            a.gslot[g_off] = s;
            a.gstart[g_off] = tok_off;
            a.gcount[g_off] = c;
            a.gitem[g_off] = i_off;
            ++g_off;
            i_off += (c + a.mts - 1) / a.mts;
        }
        cnt[s] = tok_off;                     // cursor for the placement below
        tok_off += c;
    }
    if (tid == 1023) {
        a.meta[0] = g_off;
        a.meta[1] = i_off;
        a.gitem[g_off] = i_off;
    }
    __syncthreads();

    // stable placement, tokens in order, by one wave (64 tokens per step)
    if (wv == 0) {
        for (int base = 0; base < a.T; base += 64) {
            const int t = base + lane;
            const int id = t < a.T ? a.ids[t] : -1;
            bool ok = t < a.T && id >= 0 && id < a.max_slots && a.loaded[id] != 0;
            unsigned long long act = __ballot(ok);
            while (act) {
                const int leader = __ffsll((long long)act) - 1;
                const int s = __shfl(id, leader);
                const bool mine = ok && id == s;
                const unsigned long long m = __ballot(mine);
                const int b = cnt[s];
                if (lane == leader) cnt[s] = b + __popcll(m);
                if (mine) {
                    a.perm[b + __popcll(m & ((1ull << lane) - 1ull))] = t;
                    ok = false;
                }
                act &= ~m;
            }
        }
    }
    if (tid == 0 && s_err) atomicOr(a.err, 1);
}

hipError_t launch_plan(const PlanArgs& a, hipStream_t s) {
    hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(1024), a.max_slots * sizeof(int), s, a);
    return hipGetLastError();
}

// --------------------------------------------------------------------------
// 2. shrink: Z[t, sigma * r8max + j] = scale_a * sum_k X[t, k] A_a,sigma[k, j]
// --------------------------------------------------------------------------

constexpr int kShrinkNB = 4;                  // 64 columns (rank entries) per item
constexpr int kUnroll = 2;

template <int MB>
__global__ __launch_bounds__(kThreads) void shrink_kernel(FwdArgs a) {
    constexpr int NB = kShrinkNB, MT = MB * 16, NT = NB * 16, LD = NT + 4;
    __shared__ float red[4 * MT * LD];
    const int w = threadIdx.x >> 6, l = threadIdx.x & 63, lr = l & 15, lk = (l >> 4) * 8;
    const int n_groups = a.meta[0], n_items = a.meta[1];
    const int per_proj = a.items_bound * a.cchunks;
    const int total = a.n_proj * per_proj;

    for (int flat = blockIdx.x; flat < total; flat += gridDim.x) {
        const int p = flat / per_proj, rem = flat - p * per_proj;
        const int item = rem / a.cchunks, cc = rem - item * a.cchunks;
        if (item >= n_items) continue;
        int lo = 0, hi = n_groups - 1;          // last group whose first item <= item
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (a.gitem[mid] <= item) lo = mid;
            else hi = mid - 1;
        }
        const int g = lo;
        const int slot = a.gslot[g];
        const int r8s = a.r8[slot];
        const ProjLaunch& P = a.p[p];
        const int ncols = P.n_slices * r8s;
        const int c0 = cc * NT;
        if (c0 >= ncols) continue;
        const int row0 = (item - a.gitem[g]) * MT;
        const int nrows = min(MT, a.gcount[g] - row0);
        const int* prow = a.perm + a.gstart[g] + row0;
        const uint16_t* abase = a.pool + (size_t)slot * a.slot_stride + P.a_off;

        const uint16_t* ap[MB];
        const uint16_t* bp[NB];
#pragma unroll
        for (int rb = 0; rb < MB; ++rb) {
            const int t = prow[min(rb * 16 + lr, nrows - 1)];
            ap[rb] = P.X + (size_t)t * P.K + lk;
        }
#pragma unroll
        for (int cb = 0; cb < NB; ++cb) {
            const int c = min(c0 + cb * 16 + lr, ncols - 1);
            bp[cb] = abase + (size_t)c * P.K + lk;
        }
        f32x4 acc[MB][NB];
#pragma unroll
        for (int rb = 0; rb < MB; ++rb)
#pragma unroll
            for (int cb = 0; cb < NB; ++cb) acc[rb][cb] = f32x4{0.f, 0.f, 0.f, 0.f};
        mma_ksteps<MB, NB, kUnroll>(acc, ap, bp, w * kUnroll, P.K / 32, kWaves * kUnroll);
        reduce_waves<MB, NB>(acc, red);

        const float sc = a.scale[slot];
        for (int idx = threadIdx.x; idx < MT * NT; idx += kThreads) {
            const int r = idx / NT, c = idx - (idx / NT) * NT;
            const int cg = c0 + c;
            if (r < nrows && cg < ncols) {
                const int t = prow[r];
                const int sig = cg / r8s, j = cg - sig * r8s;
                const float z = sc * red[r * LD + c];
                const uint16_t hi = f2bf(z);
                const size_t zi = (size_t)t * P.zs + sig * a.r8max + j;
                P.Z[zi] = hi;
                P.Z[zi + P.zplane] = f2bf(z - bf2f(hi));
            }
        }
        __syncthreads();
    }
}

hipError_t launch_shrink(const FwdArgs& a, int mb, hipStream_t s) {
    const int total = a.n_proj * a.items_bound * a.cchunks;
    const int grid = total < 4096 ? total : 4096;
    if (grid <= 0) return hipSuccess;
    if (mb == 1) hipLaunchKernelGGL(shrink_kernel<1>, dim3(grid), dim3(kThreads), 0, s, a);
    else hipLaunchKernelGGL(shrink_kernel<4>, dim3(grid), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

int shrink_tile_cols() { return kShrinkNB * 16; }

// --------------------------------------------------------------------------
// 3. base GEMM with fused expand
// --------------------------------------------------------------------------

template <int MB, int NB>
__global__ __launch_bounds__(kThreads) void gemm_kernel(FwdArgs a) {
    constexpr int MT = MB * 16, NT = NB * 16, LD = NT + 4;
    constexpr int kMaxOct = MT * (kMaxRank8 / 8);
    __shared__ float red[4 * MT * LD];
    __shared__ int tvid[MT];
    __shared__ unsigned bitmap[kMaxSlots / 32];
    __shared__ int oct[kMaxOct];
    __shared__ int s_noct;
    const int w = threadIdx.x >> 6, l = threadIdx.x & 63, lr = l & 15, lk = (l >> 4) * 8;

    const int bid = blockIdx.x;
    int p = 0;
    while (p + 1 < a.n_proj && bid >= a.p[p + 1].tile_base) ++p;
    const ProjLaunch& P = a.p[p];
    const int local = bid - P.tile_base;
    const int mt = local / P.tiles_n, nt = local - mt * P.tiles_n;
    const int m0 = mt * MT, n0 = nt * NT;
    const int T = a.T, N = P.N, K = P.K;

    int my_vid = -1;
    if (threadIdx.x < MT && m0 + (int)threadIdx.x < T) my_vid = a.vid[m0 + threadIdx.x];

    // ---- base product X W_s^T over this wave's k-steps
    const uint16_t* ap[MB];
    const uint16_t* bp[NB];
#pragma unroll
    for (int rb = 0; rb < MB; ++rb) {
        const int row = min(m0 + rb * 16 + lr, T - 1);
        ap[rb] = P.X + (size_t)row * K + lk;
    }
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) {
        const int col = min(n0 + cb * 16 + lr, N - 1);
        bp[cb] = P.W + (size_t)col * K + lk;
    }
    f32x4 acc[MB][NB];
#pragma unroll
    for (int rb = 0; rb < MB; ++rb)
#pragma unroll
        for (int cb = 0; cb < NB; ++cb) acc[rb][cb] = f32x4{0.f, 0.f, 0.f, 0.f};
    mma_ksteps<MB, NB, kUnroll>(acc, ap, bp, w * kUnroll, K / 32, kWaves * kUnroll);

    // ---- adapters present in this row tile, as a list of 8-rank octets
    const int nwords = (a.max_slots + 31) >> 5;
    for (int i = threadIdx.x; i < nwords; i += kThreads) bitmap[i] = 0u;
    if (threadIdx.x < MT) tvid[threadIdx.x] = my_vid;
    __syncthreads();
    if (threadIdx.x < MT && my_vid >= 0) atomicOr(&bitmap[my_vid >> 5], 1u << (my_vid & 31));
    __syncthreads();
    if (w == 0) {
        int base = 0;
        for (int wb = 0; wb < nwords; wb += 64) {
            const int wi = wb + l;
            const unsigned bits = wi < nwords ? bitmap[wi] : 0u;
            int cnt = 0;
            for (unsigned bb = bits; bb; bb &= bb - 1u) cnt += a.r8[wi * 32 + __ffs(bb) - 1] >> 3;
            int inc = cnt;
            for (int d = 1; d < 64; d <<= 1) {
                const int v = __shfl_up(inc, d);
                if (l >= d) inc += v;
            }
            int o = base + inc - cnt;
            for (unsigned bb = bits; bb; bb &= bb - 1u) {
                const int slot = wi * 32 + __ffs(bb) - 1;
                const int r8s = a.r8[slot];
                for (int j = 0; j < (r8s >> 3); ++j) oct[o++] = (slot << 12) | (r8s << 4) | j;
            }
            base += __shfl(inc, 63);
        }
        if (l == 0) s_noct = base;
    }
    __syncthreads();

    // ---- expand: acc += Zhat B over the octets (masked per token)
    const int noct = s_noct;
    const int esteps = (noct + 3) >> 2;
    int sig[NB];
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) {
        const int c = n0 + cb * 16;
        int sgm = 0;
        while (sgm + 1 < P.n_slices && c >= P.slice_col[sgm + 1]) ++sgm;
        sig[cb] = sgm;
    }
    const u32x4 zero4 = u32x4{0u, 0u, 0u, 0u};
    for (int e = w; e < esteps; e += kWaves) {
        const int o = e * 4 + (l >> 4);
        const int code = o < noct ? oct[o] : -1;
        const int slot = code >> 12, r8s = (code >> 4) & 0xff, j0 = (code & 15) * 8;
        u32x4 bv[NB];
#pragma unroll
        for (int cb = 0; cb < NB; ++cb) {
            const int col = min(n0 + cb * 16 + lr, N - 1);
            bv[cb] = code >= 0 ? ld16(a.pool + (size_t)slot * a.slot_stride + P.b_off +
                                      (size_t)col * r8s + j0)
                               : zero4;
        }
        u32x4 zh[MB], zl[MB];
#pragma unroll
        for (int cb = 0; cb < NB; ++cb) {
            if (cb == 0 || sig[cb] != sig[cb - 1]) {
#pragma unroll
                for (int rb = 0; rb < MB; ++rb) {
                    const int r = rb * 16 + lr;
                    const bool match = code >= 0 && m0 + r < T && tvid[r] == slot;
                    const uint16_t* zp = P.Z + (size_t)(m0 + r) * P.zs + sig[cb] * a.r8max + j0;
                    zh[rb] = match ? ld16(zp) : zero4;
                    zl[rb] = match ? ld16(zp + P.zplane) : zero4;
                }
            }
#pragma unroll
            for (int rb = 0; rb < MB; ++rb) {
                acc[rb][cb] = mfma(zh[rb], bv[cb], acc[rb][cb]);
                acc[rb][cb] = mfma(zl[rb], bv[cb], acc[rb][cb]);
            }
        }
    }

    // ---- reduce the 8 waves and store bf16 (two columns per thread)
    reduce_waves<MB, NB>(acc, red);
    for (int idx = threadIdx.x; idx < MT * NT / 2; idx += kThreads) {
        const int r = idx / (NT / 2), c = (idx - r * (NT / 2)) * 2;
        const int row = m0 + r, col = n0 + c;
        if (row < T && col < N) {
            const uint32_t v = (uint32_t)f2bf(red[r * LD + c]) | ((uint32_t)f2bf(red[r * LD + c + 1]) << 16);
            *reinterpret_cast<uint32_t*>(P.out + (size_t)row * N + col) = v;
        }
    }
}

int gemm_tile_rows(int mb) { return mb * 16; }
int gemm_tile_cols(int nb) { return nb * 16; }

hipError_t launch_gemm(const FwdArgs& a, int mb, int nb, hipStream_t s) {
    const dim3 grid(a.total_tiles), block(kThreads);
    if (a.total_tiles <= 0) return hipSuccess;
#define BDL_GEMM_CASE(M, NN)                                                   \
    if (mb == M && nb == NN) {                                                 \
        hipLaunchKernelGGL((gemm_kernel<M, NN>), grid, block, 0, s, a);        \
        return hipGetLastError();                                              \
    }
    BDL_GEMM_CASE(1, 1) BDL_GEMM_CASE(1, 2) BDL_GEMM_CASE(1, 4)
    BDL_GEMM_CASE(2, 1) BDL_GEMM_CASE(2, 2) BDL_GEMM_CASE(2, 4)
    BDL_GEMM_CASE(4, 1) BDL_GEMM_CASE(4, 2) BDL_GEMM_CASE(4, 4)
#undef BDL_GEMM_CASE
    return hipErrorInvalidValue;
}

// --------------------------------------------------------------------------
// adapter pack: paper layout -> kernel layout (off the per-batch path)
//   stage = [A_0 .. A_{S-1} | B_0 .. B_{S-1}],  A_s [K x r], B_s [r x n_s]
//   dst_a = A^T_cat [S * r8 x K]   (row s*r8 + j = column j of A_s, zero if j >= r)
//   dst_b = B^T_cat [N x r8]       (row n = column n of its slice's B, zero pad)
// --------------------------------------------------------------------------

struct PackArgs {
    uint16_t* dst_a;
    uint16_t* dst_b;
    const uint16_t* stage;
    int K, S, rank, r8, N;
    int slice_out[kMaxSlices];
    int slice_col[kMaxSlices + 1];
};

__global__ void pack_kernel(PackArgs a) {
    const long long na = (long long)a.S * a.r8 * a.K;
    const long long nb = (long long)a.N * a.r8;
    const long long a_elems = (long long)a.S * a.K * a.rank;
    for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < na + nb;
         i += (long long)gridDim.x * blockDim.x) {
        if (i < na) {
            const long long row = i / a.K;
            const int k = (int)(i - row * a.K);
            const int s = (int)(row / a.r8), j = (int)(row - (long long)s * a.r8);
            uint16_t v = 0;
            if (j < a.rank) v = a.stage[(long long)s * a.K * a.rank + (long long)k * a.rank + j];
            a.dst_a[i] = v;
        } else {
            const long long q = i - na;
            const int n = (int)(q / a.r8), j = (int)(q - (long long)n * a.r8);
            int s = 0;
            while (s + 1 < a.S && n >= a.slice_col[s + 1]) ++s;
            long long boff = a_elems;
            for (int u = 0; u < s; ++u) boff += (long long)a.rank * a.slice_out[u];
            uint16_t v = 0;
            if (j < a.rank) v = a.stage[boff + (long long)j * a.slice_out[s] + (n - a.slice_col[s])];
            a.dst_b[q] = v;
        }
    }
}

hipError_t launch_pack(uint16_t* dst_a, uint16_t* dst_b, const uint16_t* stage, int K, int n_slices,
                       const int* slice_out, int rank, int r8, hipStream_t s) {
    PackArgs a;
    a.dst_a = dst_a;
    a.dst_b = dst_b;
    a.stage = stage;
    a.K = K;
    a.S = n_slices;
    a.rank = rank;
    a.r8 = r8;
    int col = 0;
    for (int i = 0; i < kMaxSlices; ++i) a.slice_out[i] = i < n_slices ? slice_out[i] : 0;
    for (int i = 0; i <= kMaxSlices; ++i) {
        a.slice_col[i] = col;
        if (i < n_slices) col += slice_out[i];
    }
    a.N = col;
    const long long total = (long long)n_slices * r8 * K + (long long)col * r8;
    if (total == 0) return hipSuccess;
    long long blocks = (total + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    hipLaunchKernelGGL(pack_kernel, dim3((unsigned)blocks), dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace bdl
