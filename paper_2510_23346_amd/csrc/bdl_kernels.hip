// HIP kernels of the BD-LoRA shard forward for gfx950 (MI355X).
//
// A forward launch of one token batch over P projections (all sharing the
// tokens' adapter ids) above the decode size runs these kernels on the
// caller's stream (medium batches swap step 3 for the medium-batch GEMM and
// its epilogue in bdl_gemm.hip, large ones for the large-tile GEMM there):
//
//  1. prep_kernel   -- workgroup 0 plans the batch: validates ids and groups
//                      tokens by adapter (counting sort over slots), and
//                      writes ready-to-use work descriptors for the other two
//                      kernels (shrink items; per row tile, the adapter
//                      octets to expand).  The other workgroups copy the
//                      activations X into the MFMA fragment layout.
//  2. shrink_kernel -- Z = scale * X A for every adapter group (the LoRA
//                      "shrink", matmul_3 / matmul_5 of the paper's Fig. 2/3,
//                      step "Z <- X A" of Alg. 1 and Alg. 2).  Each group's
//                      factor A^T is streamed once; the group's token rows are
//                      gathered.
//  3. gemm_kernel   -- out = X W_s^T + Z B for each output tile: the base
//                      product (matmul_1 / matmul_2) with the LoRA "expand"
//                      (matmul_4 / matmul_6) and the add (add_1 / add_2)
//                      fused, one bf16 store per output (Alg. 1 / Alg. 2,
//                      steps "Y_adapter <- Z B" and "Y <- Y + Y_adapter").
//
// Both GEMM-shaped kernels use 8 waves per workgroup that split the K loop
// into contiguous ranges and reduce through LDS in a fixed order, so results
// are bitwise reproducible.  Their operands are read in the 1 KB fragment
// layout (see bdl_device.h).  The expand runs as extra MFMA k-steps: for the
// adapters present in the tile, 8-rank pieces ("octets") of B^T are the B
// operand and the matching Z entries (zero for tokens of other adapters) the
// A operand.  Z is kept as a pair of bf16 numbers (hi + lo, about 16
// significant bits) and multiplied in two MFMAs, so the intermediate adds no
// bf16-sized error to the LoRA term.
#include "bdl_device.h"

namespace bdl {

constexpr int kStages = 3;                    // k-steps of loads kept in flight per wave

// --------------------------------------------------------------------------
// 2. shrink: Z[t, sigma * r8max + j] = scale_a * sum_k X[t, k] A_a,sigma[k, j]
//    work item = (projection, shrink item, 16*NB-column chunk of A^T_cat)
//
//    Unsplit (shrink_kp = 1): a resident set of workgroups takes the work
//    units (projection in the order sorder, longest K first; item; chunk)
//    one at a time from a counter that the plan zeroes, so the long units
//    start first and no workgroup is spent on the host's padding of the
//    item count.
//
//    Small batches (shrink_kp = kShrinkKP): an item's adapter group holds a
//    few scattered tokens, and every item reads its rows out of the whole
//    X, so each XCD would fetch most of X from HBM.  There each item's K is
//    cut into kShrinkKP = 4 ranges, range k running on XCDs k and k + 4
//    (workgroup b runs on XCD b mod 8, and the flat index keeps the range
//    in its two low bits): each XCD fetches only its quarter of X.  (Eight
//    ranges, one per XCD, leave each wave too few k-steps to stream.)  The
//    ranges store fp32 partial tiles (their own workspace);
//    shrink_reduce_kernel adds them in range order and writes Z.
// --------------------------------------------------------------------------

// XRM: the launch's projections read the caller's row-major X (the
// large-tile path); else the packed X
template <int MB, int NB, bool XRM>
__global__ __launch_bounds__(kThreads) void shrink_kernel(FwdArgs a) {
    constexpr int MT = MB * 16, NT = NB * 16, FR = MB * NB * 64;
    // the waves' sums in lane order (fragment (rb, cb) of wave w at
    // ((w MB + rb) NB + cb) 64 + lane), added in wave order after one barrier
    __shared__ f32x4 red[kWaves * FR];
    const int w = wave_id(), l = threadIdx.x & 63, lr = l & 15;
    // (clamped: the plan writes at most items_bound items)
    const int n_items = min(a.meta[1], a.items_bound);
    const int KP = a.shrink_kp;
    const bool queue = KP == 1;
    const int per_proj = (queue ? n_items : a.items_bound) * a.cchunks;
    const int total = a.n_proj * per_proj * KP;
    __shared__ int s_unit;

    for (int iter = 0;; ++iter) {
        int flat = blockIdx.x + iter * gridDim.x;
        if (queue) {
            if (threadIdx.x == 0) s_unit = atomicAdd(a.queue, 1);
            __syncthreads();
            flat = s_unit;
            __syncthreads();
        }
        if (flat >= total) break;
        const int f = flat / KP, kp = flat - f * KP;
        const int ps = f / per_proj, rem = f - ps * per_proj;
        const int p = queue ? a.sorder[ps] : ps;
        const int item = rem / a.cchunks, cc = rem - item * a.cchunks;
        const int4 it = a.items[item];       // in bounds for every item < items_bound
        if (item >= n_items) continue;
        const int slot = it.x, nrows = it.z, r8s = it.w;
        const ProjLaunch& P = a.p[p];
        const int ncols = P.n_slices * r8s;
        const int c0 = cc * NT;
        if (c0 >= ncols) continue;
        const float sc = a.scale[slot];
        const int* prow = a.perm + it.y;
        const int KS = P.K >> 5;
        const int nblk = (ncols + 15) >> 4;
        const uint16_t* abase = a.pool + (size_t)slot * a.slot_stride + P.a_off;

        // the lane's row (token t) at k-step 0: in X row-major (k-steps 32
        // elements apart) or in the packed X (k-steps a fragment apart)
        const uint16_t* ap[MB];
        const uint16_t* bp[NB];
#pragma unroll
        for (int rb = 0; rb < MB; ++rb) {
            const int t = prow[min(rb * 16 + lr, nrows - 1)];
            ap[rb] = XRM ? P.X + (size_t)t * P.K + 8 * (l >> 4)
                         : P.Xp + frag_index(t >> 4, 0, KS) + ((t & 15) + 16 * (l >> 4)) * 8;
        }
#pragma unroll
        for (int cb = 0; cb < NB; ++cb) bp[cb] = abase + frag_index(min((c0 >> 4) + cb, nblk - 1), 0, KS) + l * 8;
        f32x4 acc[MB][NB];
#pragma unroll
        for (int rb = 0; rb < MB; ++rb)
#pragma unroll
            for (int cb = 0; cb < NB; ++cb) acc[rb][cb] = f32x4{0.f, 0.f, 0.f, 0.f};
        // this range's k-steps, split over the 8 waves
        const int ks0 = kp * KS / KP;
        int k0, nk;
        wave_krange((kp + 1) * KS / KP - ks0, w, &k0, &nk);
        if (nk > 0) mma_range<MB, NB, kStages>(acc, ap, bp, ks0 + k0, nk, XRM ? 32 : kFrag, kFrag);
#pragma unroll
        for (int rb = 0; rb < MB; ++rb)
#pragma unroll
            for (int cb = 0; cb < NB; ++cb) red[((w * MB + rb) * NB + cb) * 64 + l] = acc[rb][cb];
        __syncthreads();
        // thread = one fragment slot at a time: rows rb 16 + 4 (ln / 16) + i
        // (i < 4), column cb 16 + ln mod 16
        float* const part = a.shrinkpart + (size_t)flat * (MT * NT);
        for (int e = threadIdx.x; e < FR; e += kThreads) {
            f32x4 v = red[e];
#pragma unroll
            for (int ww = 1; ww < kWaves; ++ww) v += red[ww * FR + e];
            const int fr = e >> 6, ln = e & 63, rb = fr / NB, cb = fr - rb * NB;
            const int c = cb * 16 + (ln & 15), cg = c0 + c;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int r = rb * 16 + 4 * (ln >> 4) + i;
                if (KP > 1) {
                    // partial tile of range kp (row-major MT x NT), summed by shrink_reduce_kernel
                    part[r * NT + c] = v[i];
                } else if (r < nrows && cg < ncols) {
                    const int t = prow[r];
                    const int sig = cg / r8s, j = cg - sig * r8s;
                    const float z = sc * v[i];
                    const uint16_t hi = f2bf(z);
                    const size_t zi = (size_t)t * P.zs + sig * a.r8max + j;
                    P.Z[zi] = hi;
                    P.Z[zi + P.zplane] = f2bf(z - bf2f(hi));
                }
            }
        }
        __syncthreads();
    }
}

// Z of the split shrink: the kShrinkKP range partials of each (projection,
// item, chunk) tile added in range order, scaled, stored as the bf16 pair.
template <int MB, int NB>
__global__ __launch_bounds__(256) void shrink_reduce_kernel(FwdArgs a) {
    constexpr int MT = MB * 16, NT = NB * 16, KP = kShrinkKP;
    const int n_items = a.meta[1];
    const int per_proj = a.items_bound * a.cchunks;
    const int total = a.n_proj * per_proj;
    for (int f = blockIdx.x; f < total; f += gridDim.x) {
        const int p = f / per_proj, rem = f - p * per_proj;
        const int item = rem / a.cchunks, cc = rem - item * a.cchunks;
        const int4 it = a.items[item];
        if (item >= n_items) continue;
        const int slot = it.x, nrows = it.z, r8s = it.w;
        const ProjLaunch& P = a.p[p];
        const int ncols = P.n_slices * r8s, c0 = cc * NT;
        if (c0 >= ncols) continue;
        const float sc = a.scale[slot];
        const int* prow = a.perm + it.y;
        const float* src = a.shrinkpart + (size_t)f * KP * (MT * NT);
        for (int idx = threadIdx.x; idx < MT * NT; idx += 256) {
            const int r = idx / NT, c = idx - (idx / NT) * NT, cg = c0 + c;
            if (r < nrows && cg < ncols) {
                float z = 0.f;
#pragma unroll
                for (int k = 0; k < KP; ++k) z += src[(size_t)k * (MT * NT) + idx];
                z *= sc;
                const int t = prow[r];
                const int sig = cg / r8s, j = cg - sig * r8s;
                const uint16_t hi = f2bf(z);
                const size_t zi = (size_t)t * P.zs + sig * a.r8max + j;
                P.Z[zi] = hi;
                P.Z[zi + P.zplane] = f2bf(z - bf2f(hi));
            }
        }
    }
}

// workgroups of the shrink kernel that the device holds at once (cached)
template <int MB, int NB, bool XRM>
int shrink_resident() {
    static int n = 0;
    if (n == 0) {
        int dev = 0, cu = 0, per = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, shrink_kernel<MB, NB, XRM>, kThreads, 0) != hipSuccess)
            return 0;
        n = cu * (per > 1 ? per : 1);
    }
    return n;
}

hipError_t launch_shrink(const FwdArgs& a, int mb, int nb, hipStream_t s) {
    const int KP = a.shrink_kp;
    if (KP != 1 && (KP != kShrinkKP || !a.shrinkpart)) return hipErrorInvalidValue;
    if (KP == 1 && !a.queue) return hipErrorInvalidValue;
    for (int i = 0; i < a.n_proj; ++i)
        if (a.sorder[i] < 0 || a.sorder[i] >= a.n_proj) return hipErrorInvalidValue;
    const int tiles = a.n_proj * a.items_bound * a.cchunks;
    const int total = tiles * KP;
    // split: every unit at once, or a multiple of 8 workgroups (either way
    // each workgroup keeps one k-range, so XCD b mod 8 gets range b mod 4);
    // unsplit: the resident workgroups take units from the queue
    const int cap = 4096;
    if (total <= 0) return hipSuccess;
    const int rgrid = tiles < 2048 ? tiles : 2048;
    // every projection of a launch reads X the same way (the large-tile path
    // reads the caller's row-major X)
    const bool xrm = a.p[0].x_rowmajor != 0;
    for (int i = 1; i < a.n_proj; ++i)
        if ((a.p[i].x_rowmajor != 0) != xrm) return hipErrorInvalidValue;
#define BDL_SHRINK_LAUNCH(M, NN, X)                                                                 \
    {                                                                                               \
        int grid = total < cap ? total : cap;                                                       \
        if (KP == 1) {                                                                              \
            const int r = shrink_resident<M, NN, X>();                          \
            if (r <= 0) return hipErrorInvalidValue;                                                \
            grid = total < r ? total : r;                                                           \
        }                                                                                           \
        hipLaunchKernelGGL((shrink_kernel<M, NN, X>), dim3(grid), dim3(kThreads), 0, s, a);         \
    }
#define BDL_SHRINK_CASE(M, NN)                                                                          \
    if (mb == M && nb == NN) {                                                                          \
        if (xrm)                                                                                        \
            BDL_SHRINK_LAUNCH(M, NN, true)                                                              \
        else                                                                                            \
            BDL_SHRINK_LAUNCH(M, NN, false)                                                             \
        if (KP > 1) hipLaunchKernelGGL((shrink_reduce_kernel<M, NN>), dim3(rgrid), dim3(256), 0, s, a); \
        return hipGetLastError();                                                                       \
    }
    BDL_SHRINK_CASE(1, 1) BDL_SHRINK_CASE(1, 2) BDL_SHRINK_CASE(1, 4)
    BDL_SHRINK_CASE(4, 1) BDL_SHRINK_CASE(4, 2) BDL_SHRINK_CASE(4, 4) BDL_SHRINK_CASE(2, 6)
#undef BDL_SHRINK_CASE
#undef BDL_SHRINK_LAUNCH
    return hipErrorInvalidValue;
}

// --------------------------------------------------------------------------
// 3. base GEMM with fused expand
// --------------------------------------------------------------------------

template <int MB, int NB>
__global__ __launch_bounds__(kThreads) void gemm_kernel(FwdArgs a) {
    constexpr int MT = MB * 16, NT = NB * 16, LD = NT + 4;
    __shared__ float red[4 * MT * LD];
    const int w = wave_id(), l = threadIdx.x & 63, lr = l & 15;

    const int bid = blockIdx.x;
    int p = 0;
    while (p + 1 < a.n_proj && bid >= a.p[p + 1].tile_base) ++p;
    const ProjLaunch& P = a.p[p];
    const int local = bid - P.tile_base;
    const int mt = local / P.tiles_n, nt = local - mt * P.tiles_n;
    const int m0 = mt * MT, n0 = nt * NT;
    const int T = a.T, N = P.N, K = P.K;

    // expand inputs that do not depend on the base product: fetched first
    const int* codes = a.tile_oct + (size_t)mt * a.oct_cap;
    int code = codes[4 * w + (l >> 4)];
    int rvid[MB];
#pragma unroll
    for (int rb = 0; rb < MB; ++rb) {
        const int row = m0 + rb * 16 + lr;
        rvid[rb] = row < T ? a.vid[row] : -1;
    }

    // ---- base product X W_s^T over this wave's k-steps
    const int KS = K >> 5;
    const int nrb = (T + 15) >> 4, ncb = N >> 4;
    const uint16_t* ap[MB];
    const uint16_t* bp[NB];
#pragma unroll
    for (int rb = 0; rb < MB; ++rb) ap[rb] = P.Xp + frag_index(min(mt * MB + rb, nrb - 1), 0, KS) + l * 8;
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) bp[cb] = P.W + frag_index(min(nt * NB + cb, ncb - 1), 0, KS) + l * 8;
    f32x4 acc[MB][NB];
#pragma unroll
    for (int rb = 0; rb < MB; ++rb)
#pragma unroll
        for (int cb = 0; cb < NB; ++cb) acc[rb][cb] = f32x4{0.f, 0.f, 0.f, 0.f};
    int k0, nk;
    wave_krange(KS, w, &k0, &nk);
    if (P.Ws) {
        // INT4 base: same tile, the raw q on the matrix cores, scales in fp32
        const char* wq[NB];
        const uint16_t* wsc[NB];
#pragma unroll
        for (int cb = 0; cb < NB; ++cb) {
            const int blk = min(nt * NB + cb, ncb - 1);
            wq[cb] = reinterpret_cast<const char*>(P.W) + (size_t)blk * KS * kInt4FragBytes + l * 4;
            wsc[cb] = P.Ws + (size_t)blk * (KS / kInt4Group) * 16 + lr;
        }
        if (nk > 0) mma_range_int4<MB, NB, kStages>(acc, ap, wq, wsc, k0, nk);
    } else if (nk > 0) {
        mma_range<MB, NB, kStages>(acc, ap, bp, k0, nk, kFrag, kFrag);
    }

    // ---- expand: acc += Zhat B over the tile's octets (masked per token)
    int sig[NB];
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) {
        const int c = n0 + cb * 16;
        int sgm = 0;
        while (sgm + 1 < P.n_slices && c >= P.slice_col[sgm + 1]) ++sgm;
        sig[cb] = sgm;
    }
    const u32x4 zero4 = u32x4{0u, 0u, 0u, 0u};
    for (int e = w;;) {
        if (!__any(code >= 0)) break;
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
                    const bool match = code >= 0 && rvid[rb] == slot;
                    const uint16_t* zp = P.Z + (size_t)(m0 + rb * 16 + lr) * P.zs + sig[cb] * a.r8max + j0;
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
        e += kWaves;
        if (4 * e + 4 > a.oct_cap) break;
        code = codes[4 * e + (l >> 4)];
    }

    // ---- reduce the 8 waves and store bf16 (or fp32), two columns per thread
    reduce_waves<MB, NB>(acc, red);
    for (int idx = threadIdx.x; idx < MT * NT / 2; idx += kThreads) {
        const int r = idx / (NT / 2), c = (idx - r * (NT / 2)) * 2;
        const int row = m0 + r, col = n0 + c;
        if (row < T && col < N) {
            if (P.out_f32) {
                *reinterpret_cast<float2*>(P.out_f32 + (size_t)row * N + col) =
                    float2{red[r * LD + c], red[r * LD + c + 1]};
            } else {
                const uint32_t v = (uint32_t)f2bf(red[r * LD + c]) | ((uint32_t)f2bf(red[r * LD + c + 1]) << 16);
                *reinterpret_cast<uint32_t*>(P.out + (size_t)row * N + col) = v;
            }
        }
    }
}

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
// packing (off the per-batch path)
// --------------------------------------------------------------------------

// rows-major [rows x K] -> fragment layout with rows padded to 16 (zeros)
__global__ void pack_rows_kernel(const uint16_t* src, uint16_t* dst, int rows, int K, long long frags) {
    const int l = threadIdx.x & 63;
    const int KS = K >> 5;
    for (long long f = (blockIdx.x * (long long)blockDim.x + threadIdx.x) >> 6; f < frags;
         f += ((long long)gridDim.x * blockDim.x) >> 6) {
        const int rb = (int)(f / KS), ks = (int)(f - (long long)rb * KS);
        const int row = rb * 16 + (l & 15);
        u32x4 v = u32x4{0u, 0u, 0u, 0u};
        if (row < rows) v = ld16(src + (size_t)row * K + ks * 32 + (l >> 4) * 8);
        *reinterpret_cast<u32x4*>(dst + (size_t)f * kFrag + l * 8) = v;
    }
}

hipError_t launch_pack_rows(const uint16_t* src, uint16_t* dst, int rows, int K, hipStream_t s) {
    const long long frags = (long long)((rows + 15) / 16) * (K / 32);
    if (frags == 0) return hipSuccess;
    long long blocks = (frags + 3) / 4;
    if (blocks > 16384) blocks = 16384;
    hipLaunchKernelGGL(pack_rows_kernel, dim3((unsigned)blocks), dim3(256), 0, s, src, dst, rows, K, frags);
    return hipGetLastError();
}

// INT4 base weight: nn.Linear rows of nibbles (low nibble = even input) and
// bf16 scales [N x K/128] -> the forward layout (one 32-bit word per lane and
// k-step, then the scales grouped per 16-column block).  Thread = one word or
// one scale.
__global__ void pack_int4_kernel(const uint8_t* q, const uint16_t* scales, uint32_t* dst_w, uint16_t* dst_s, int N,
                                 int K) {
    const long long words = (long long)N * K / 8, nsc = (long long)N * (K / 128);
    const int KS = K >> 5, G = K >> 7;
    for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < words + nsc;
         i += (long long)gridDim.x * blockDim.x) {
        if (i < words) {
            const int l = (int)(i & 63);
            const long long f = i >> 6;
            const int rb = (int)(f / KS), ks = (int)(f - (long long)rb * KS);
            const int n = rb * 16 + (l & 15), k0 = ks * 32 + (l >> 4) * 8;
            const uint8_t* src = q + (size_t)n * (K / 2) + k0 / 2;
            uint32_t w = 0;
#pragma unroll
            for (int v = 0; v < 8; ++v) {
                const uint32_t nib = (src[v >> 1] >> (4 * (v & 1))) & 15u;
                w |= nib << (4 * (v >> 1) + 16 * (v & 1));
            }
            dst_w[i] = w;
        } else {
            const long long j = i - words;
            const int c = (int)(j & 15);
            const long long r = j >> 4;
            const int rb = (int)(r / G), g = (int)(r - (long long)rb * G);
            dst_s[j] = scales[(size_t)(rb * 16 + c) * G + g];
        }
    }
}

hipError_t launch_pack_int4(const uint8_t* q, const uint16_t* scales, uint32_t* dst_w, uint16_t* dst_s, int N,
                            int K, hipStream_t s) {
    const long long total = (long long)N * K / 8 + (long long)N * (K / 128);
    if (total == 0) return hipSuccess;
    long long blocks = (total + 255) / 256;
    if (blocks > 16384) blocks = 16384;
    hipLaunchKernelGGL(pack_int4_kernel, dim3((unsigned)blocks), dim3(256), 0, s, q, scales, dst_w, dst_s, N, K);
    return hipGetLastError();
}

// slot tables of consecutive adapter slots, written in stream order after
// their slabs
__global__ void set_slots_kernel(int* r8, float* scale, int* loaded, SlotBatch b) {
    const int i = threadIdx.x;
    if (i < b.n) {
        r8[b.first + i] = b.r8[i];
        scale[b.first + i] = b.scale[i];
        loaded[b.first + i] = 1;
    }
}

hipError_t launch_set_slots(int* r8, float* scale, int* loaded, const SlotBatch& b, hipStream_t s) {
    if (b.n < 1 || b.n > kMaxSlotBatch) return hipErrorInvalidValue;
    hipLaunchKernelGGL(set_slots_kernel, dim3(1), dim3(64), 0, s, r8, scale, loaded, b);
    return hipGetLastError();
}

// adapter: paper layout -> pool layout
//   stage = [A_0 .. A_{S-1} | B_0 .. B_{S-1}],  A_s [K x r], B_s [r x n_s]
//   dst_a = A^T_cat in fragment layout: row s*r8 + j of A^T_cat is column j
//           of A_s (zero for j >= r), rows padded to a multiple of 16
//   dst_b = B^T_cat [N x r8] row-major: row n is column n of its slice's B
struct PackArgs {
    uint16_t* dst_a;
    uint16_t* dst_b;
    const uint16_t* stage;
    int K, S, rank, r8, N;
    int slice_out[kMaxSlices];
    int slice_col[kMaxSlices + 1];
};

__global__ void pack_adapter_kernel(PackArgs a) {
    const int KS = a.K >> 5;
    const int arows = a.S * a.r8;
    const long long na = (long long)((arows + 15) / 16) * KS * kFrag;
    const long long nb = (long long)a.N * a.r8;
    const long long a_elems = (long long)a.S * a.K * a.rank;
    for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < na + nb;
         i += (long long)gridDim.x * blockDim.x) {
        if (i < na) {
            const long long f = i / kFrag;
            const int e = (int)(i - f * kFrag), l = e >> 3, q = e & 7;
            const int rb = (int)(f / KS), ks = (int)(f - (long long)rb * KS);
            const int row = rb * 16 + (l & 15), k = ks * 32 + (l >> 4) * 8 + q;
            uint16_t v = 0;
            if (row < arows) {
                const int s = row / a.r8, j = row - s * a.r8;
                if (j < a.rank) v = a.stage[(long long)s * a.K * a.rank + (long long)k * a.rank + j];
            }
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

hipError_t launch_pack_adapter(uint16_t* dst_a, uint16_t* dst_b, const uint16_t* stage, int K, int n_slices,
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
    const long long total = (long long)((n_slices * r8 + 15) / 16) * (K / 32) * kFrag + (long long)col * r8;
    if (total == 0) return hipSuccess;
    long long blocks = (total + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    hipLaunchKernelGGL(pack_adapter_kernel, dim3((unsigned)blocks), dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace bdl
