// C ABI of the BD-LoRA shard library: adapter pool, validation, host plan,
// and the forward launch sequence (plan -> shrink -> base GEMM + expand).
#include "bdlora.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <string>
#include <vector>

#include "bdl_launch.h"

namespace {

thread_local std::string g_err;

int fail(int code, const std::string& msg) {
    g_err = msg;
    return code;
}

#define BDL_HIP(expr)                                                                        \
    do {                                                                                     \
        hipError_t e_ = (expr);                                                              \
        if (e_ != hipSuccess) return fail(BDLORA_ERR_HIP, std::string(#expr) + ": " + hipGetErrorString(e_)); \
    } while (0)

constexpr long long kAlign = 128;  // elements (256 bytes)
constexpr int kProfEvents = 8;     // timing events per profiled forward: 4 intervals

long long round_up(long long v, long long m) { return (v + m - 1) / m * m; }
int rank8(int r) { return (r + 7) / 8 * 8; }

struct ProjInfo {
    int kind, K, S, N, zs;
    int wfmt;                         // BDLORA_WEIGHT_*
    int slice_out[bdl::kMaxSlices];
    int slice_col[bdl::kMaxSlices + 1];
    long long a_off, b_off;           // element offsets inside a slot
};

struct Layout {
    int n_projs = 0;
    ProjInfo proj[bdl::kMaxProjs];
    int max_slots = 0, max_rank = 0, r8max = 0, max_tokens = 0;
    long long slot_stride = 0;         // elements
    long long slab_bytes = 0, ws_bytes = 0;
    long long z_elems[bdl::kMaxProjs];
    long long xp_elems[bdl::kMaxProjs];
    long long part_slots = 0;          // decode partial tiles
    long long mlp_elems = 0;           // prefill MLP: gate and up outputs, fp32
    long long bigpart_elems = 0;       // large-tile GEMM: fp32 partials of split tiles
    long long shrinkpart_elems = 0;    // split shrink: fp32 partials
};

// Validates the pool arguments and computes the memory layout.
int make_layout(const bdlora_proj_desc* projs, int n_projs, int max_slots, int max_rank,
                int max_tokens, Layout* L) {
    if (!projs || !L) return fail(BDLORA_ERR_INVALID_ARG, "null projection list");
    if (n_projs < 1 || n_projs > BDLORA_MAX_PROJS)
        return fail(BDLORA_ERR_INVALID_ARG, "n_projs must be 1..8");
    if (max_slots < 1 || max_slots > BDLORA_MAX_SLOTS)
        return fail(BDLORA_ERR_INVALID_ARG, "max_slots must be 1..8192");
    if (max_rank < 0 || max_rank > BDLORA_MAX_RANK)
        return fail(BDLORA_ERR_INVALID_ARG, "max_rank must be 0..128");
    if (max_tokens < 1 || max_tokens > (1 << 24))
        return fail(BDLORA_ERR_INVALID_ARG, "max_tokens must be 1..16777216");
    L->n_projs = n_projs;
    L->max_slots = max_slots;
    L->max_rank = max_rank;
    L->r8max = std::max(8, rank8(max_rank));
    L->max_tokens = max_tokens;
    long long off = 0;
    for (int p = 0; p < n_projs; ++p) {
        const bdlora_proj_desc& d = projs[p];
        ProjInfo& P = L->proj[p];
        if (d.kind != BDLORA_COLUMN && d.kind != BDLORA_ROW)
            return fail(BDLORA_ERR_INVALID_ARG, "projection kind must be COLUMN or ROW");
        if (d.d_in < 32 || d.d_in % 32 || d.d_in > (1 << 20))
            return fail(BDLORA_ERR_SHAPE, "d_in must be a positive multiple of 32");
        if (d.n_slices < 1 || d.n_slices > BDLORA_MAX_SLICES)
            return fail(BDLORA_ERR_SHAPE, "n_slices must be 1..4");
        P.kind = d.kind;
        P.K = d.d_in;
        P.S = d.n_slices;
        int col = 0;
        for (int s = 0; s < bdl::kMaxSlices; ++s) {
            P.slice_out[s] = s < d.n_slices ? d.slice_out[s] : 0;
            P.slice_col[s] = col;
            if (s < d.n_slices) {
                if (d.slice_out[s] < 16 || d.slice_out[s] % 16 || d.slice_out[s] > (1 << 20))
                    return fail(BDLORA_ERR_SHAPE, "slice_out must be a positive multiple of 16");
                col += d.slice_out[s];
            }
        }
        P.slice_col[bdl::kMaxSlices] = col;
        for (int s = d.n_slices; s <= bdl::kMaxSlices; ++s) P.slice_col[s] = col;
        P.N = col;
        if (d.weight_format != BDLORA_WEIGHT_BF16 && d.weight_format != BDLORA_WEIGHT_INT4_G128)
            return fail(BDLORA_ERR_INVALID_ARG, "unknown weight_format");
        if (d.weight_format == BDLORA_WEIGHT_INT4_G128 && (P.K % 128 || P.N % 64))
            return fail(BDLORA_ERR_SHAPE, "an INT4 base needs d_in a multiple of 128 and d_out a multiple of 64");
        P.wfmt = d.weight_format;
        P.zs = P.S * L->r8max;
        P.a_off = off;                                   // packed A^T_cat, rows padded to 16
        off = round_up(off + round_up((long long)P.S * L->r8max, 16) * P.K, kAlign);
        P.b_off = off;
        off = round_up(off + (long long)P.N * L->r8max, kAlign);
        L->z_elems[p] = 2LL * max_tokens * P.zs;      // hi and lo planes
        L->xp_elems[p] = round_up(max_tokens, 16) * P.K;
    }
    L->slot_stride = off;
    L->slab_bytes = (long long)max_slots * off * 2;
    long long ws = 0;
    ws += 9LL * max_tokens * 4;                                   // vid, tr8, tgrp, perm, rowtok, rowslot (+ slack)
    ws += 4LL * (max_slots + 2) * 4 + 2 * 4;                      // group tables, meta, err
    ws += ((long long)max_slots + max_tokens / 16 + 2) * 16;      // shrink items
    ws += std::max(((long long)max_tokens / 16 + 1) * (2LL * L->r8max + 64),
                   ((long long)max_tokens / 64 + 1) * (8LL * L->r8max + 64)) * 4;   // tile octets
    for (int p = 0; p < n_projs; ++p) ws += (L->z_elems[p] + L->xp_elems[p]) * 2;
    // decode partial tiles: one per (group, workgroup) pair of the main launch
    long long groups = 0;
    const int act_max = std::min({bdl::kDecodeMaxT, max_slots, max_tokens});
    for (int p = 0; p < n_projs; ++p) {
        const ProjInfo& P = L->proj[p];
        groups += (P.N / 16 + (long long)act_max * ((P.S * L->r8max + 15) / 16) + 3) / 4;
    }
    L->part_slots = groups + bdl::kDecMaxGrid;
    ws += L->part_slots * bdl::kPartElems * 4 + (long long)max_tokens * 4;
    int max_n = 0;                                  // widest single-slice column projection
    for (int p = 0; p < n_projs; ++p)
        if (L->proj[p].kind == BDLORA_COLUMN && L->proj[p].S == 1) max_n = std::max(max_n, L->proj[p].N);
    L->mlp_elems = 2LL * max_tokens * max_n;
    ws += L->mlp_elems * 4;
    // fp32 partials of the large-tile GEMM's split tiles (pools for batches
    // above the decode size)
    L->bigpart_elems = max_tokens > bdl::kDecodeMaxT ? (long long)bdl::kBigPartSlots * bdl::kBigPartElems : 0;
    ws += L->bigpart_elems * 4;
    // and of the split shrink (which can run beside the base product)
    L->shrinkpart_elems = max_tokens > bdl::kDecodeMaxT ? bdl::kShrinkPartElems : 0;
    ws += L->shrinkpart_elems * 4;
    ws += max_slots * 12LL;                                       // slot tables
    L->ws_bytes = ws;
    return BDLORA_OK;
}

struct DeviceGuard {
    int old = -1;
    bool ok = false;
    explicit DeviceGuard(int dev) {
        if (hipGetDevice(&old) == hipSuccess && hipSetDevice(dev) == hipSuccess) ok = true;
    }
    ~DeviceGuard() {
        if (old >= 0) (void)hipSetDevice(old);
    }
};

// The adapters of a batch as the forward got them: device ids, or host
// segments validated and copied here (they travel with the prep launch).
struct Batch {
    const int32_t* ids = nullptr;     // device [T], or null
    int n_seg = 0;
    int seg_start[bdl::kMaxSeg];
    int seg_slot[bdl::kMaxSeg];
};

}  // namespace

struct bdlora_pool {
    int device = 0;
    Layout L;
    uint16_t* d_slabs = nullptr;
    int* d_r8 = nullptr;
    float* d_scale = nullptr;
    int* d_loaded = nullptr;
    std::vector<int> h_rank, h_r8, h_loaded;
    std::vector<float> h_scale;
    int* d_vid = nullptr;
    int* d_tr8 = nullptr;
    int* d_perm = nullptr;
    int* d_gslot = nullptr;
    int* d_gr8 = nullptr;
    int* d_gstart = nullptr;
    int* d_gcount = nullptr;
    int4* d_items = nullptr;
    int* d_tile_oct = nullptr;
    int* d_rowtok = nullptr;
    int* d_rowslot = nullptr;
    long long items_cap = 0, oct_elems = 0;
    int* d_meta = nullptr;
    int* d_err = nullptr;
    uint16_t* d_Z[bdl::kMaxProjs] = {};
    int* d_tgrp = nullptr;
    float* d_part = nullptr;
    float* d_mlp = nullptr;
    float* d_bigpart = nullptr;
    float* d_shrinkpart = nullptr;
    // medium batches: the shrink runs on side_stream, forked from the
    // caller's stream after the prep launch and joined back before the
    // epilogue
    hipStream_t side_stream = nullptr;
    hipEvent_t fork_ev = nullptr, join_ev = nullptr;
    int n_cu = 0;
    uint16_t* d_Xp[bdl::kMaxProjs] = {};
    uint16_t* d_stage = nullptr;
    long long stage_elems = 0;
    hipStream_t load_stream = nullptr;
    long long bytes = 0;
    // timing hooks
    int prof_left = 0;
    int prof_used = 0;
    int last_path = 0;        // BDLORA_PATH_* of the last forward
    hipError_t static_err = hipSuccess;   // taking the static scratch's address at creation
    std::vector<hipEvent_t> prof_ev;      // kProfEvents per recorded call
};

namespace {

void free_pool(bdlora_pool* P) {
    if (!P) return;
    auto f = [](void* p) {
        if (p) (void)hipFree(p);
    };
    f(P->d_slabs);
    f(P->d_r8);
    f(P->d_scale);
    f(P->d_loaded);
    f(P->d_vid);
    f(P->d_tr8);
    f(P->d_perm);
    f(P->d_gslot);
    f(P->d_gr8);
    f(P->d_gstart);
    f(P->d_gcount);
    f(P->d_items);
    f(P->d_tile_oct);
    f(P->d_rowtok);
    f(P->d_rowslot);
    f(P->d_meta);
    f(P->d_err);
    for (auto z : P->d_Z) f(z);
    f(P->d_tgrp);
    f(P->d_part);
    f(P->d_mlp);
    f(P->d_bigpart);
    f(P->d_shrinkpart);
    for (auto x : P->d_Xp) f(x);
    f(P->d_stage);
    for (auto e : P->prof_ev) (void)hipEventDestroy(e);
    if (P->load_stream) (void)hipStreamDestroy(P->load_stream);
    if (P->side_stream) (void)hipStreamDestroy(P->side_stream);
    if (P->fork_ev) (void)hipEventDestroy(P->fork_ev);
    if (P->join_ev) (void)hipEventDestroy(P->join_ev);
    delete P;
}

template <typename T>
int dev_alloc(T** p, long long elems, long long* total) {
    const size_t bytes = (size_t)std::max(1LL, elems) * sizeof(T);
    hipError_t e = hipMalloc((void**)p, bytes);
    if (e != hipSuccess) {
        *p = nullptr;
        (void)hipGetLastError();
        return fail(e == hipErrorOutOfMemory ? BDLORA_ERR_OOM : BDLORA_ERR_HIP,
                    std::string("hipMalloc of ") + std::to_string(bytes) + " bytes: " + hipGetErrorString(e));
    }
    *total += (long long)bytes;
    return BDLORA_OK;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

}  // namespace

namespace {

// Pack one adapter into the slot layout of L (host memory, slot_stride
// elements, padding zeroed): the work of bdlora_pack_adapter_host.
int pack_adapter_slab(const Layout& L, int rank, const uint16_t* const* A_host, const uint16_t* const* B_host,
                      uint16_t* slab) {
    if (rank < 0 || rank > L.max_rank) return fail(BDLORA_ERR_INVALID_ARG, "rank out of range 0..max_rank");
    if (rank > 0 && (!A_host || !B_host)) return fail(BDLORA_ERR_INVALID_ARG, "null factor arrays");
    const int r8 = rank8(rank);
    std::memset(slab, 0, (size_t)L.slot_stride * 2);
    int k = 0;
    for (int p = 0; p < L.n_projs; ++p) {
        const ProjInfo& pi = L.proj[p];
        if (rank == 0) {
            k += pi.S;
            continue;
        }
        for (int s = 0; s < pi.S; ++s) {
            if (!A_host[k + s] || !B_host[k + s]) return fail(BDLORA_ERR_INVALID_ARG, "null factor pointer");
        }
        // A^T_cat in the fragment layout: row s*r8 + j is column j of A_s
        // (zero for j >= rank), rows padded to 16; element
        // [(rb KS + ks) 512 + lane 8 + i] = A^T_cat[16 rb + lane%16][32 ks + 8 (lane/16) + i]
        const int KS = pi.K / 32, arows = pi.S * r8;
        uint16_t* da = slab + pi.a_off;
        for (int row = 0; row < arows; ++row) {
            const int s = row / r8, j = row - s * r8;
            if (j >= rank) continue;
            const uint16_t* a = A_host[k + s];
            const int rb = row / 16, lr = row % 16;
            for (int kk = 0; kk < pi.K; ++kk) {
                const uint16_t v = a[(size_t)kk * rank + j];
                if ((v & 0x7f80u) == 0x7f80u) return fail(BDLORA_ERR_INVALID_ARG, "non-finite value in A");
                const int ks = kk / 32, w = kk % 32, lane = lr + 16 * (w / 8), i = w % 8;
                da[((size_t)rb * KS + ks) * 512 + lane * 8 + i] = v;
            }
        }
        // B^T_cat [N x r8] row-major: row n is column n of its slice's B
        uint16_t* db = slab + pi.b_off;
        for (int s = 0; s < pi.S; ++s) {
            const uint16_t* b = B_host[k + s];
            const int n_s = pi.slice_out[s];
            for (int j = 0; j < rank; ++j)
                for (int n = 0; n < n_s; ++n) {
                    const uint16_t v = b[(size_t)j * n_s + n];
                    if ((v & 0x7f80u) == 0x7f80u) return fail(BDLORA_ERR_INVALID_ARG, "non-finite value in B");
                    db[(size_t)(pi.slice_col[s] + n) * r8 + j] = v;
                }
        }
        k += pi.S;
    }
    return BDLORA_OK;
}

}  // namespace

extern "C" {

const char* bdlora_last_error(void) { return g_err.c_str(); }

int bdlora_layout_slot_bytes(const bdlora_proj_desc* projs, int32_t n_projs, int32_t max_rank, int64_t* bytes) {
    if (!bytes) return fail(BDLORA_ERR_INVALID_ARG, "null output");
    Layout L;
    int rc = make_layout(projs, n_projs, 1, max_rank, 1, &L);
    if (rc) return rc;
    *bytes = L.slot_stride * 2;
    return BDLORA_OK;
}

int bdlora_pack_adapter_layout(const bdlora_proj_desc* projs, int32_t n_projs, int32_t max_rank, int32_t rank,
                               const uint16_t* const* A_host, const uint16_t* const* B_host, void* slab_host) {
    if (!slab_host) return fail(BDLORA_ERR_INVALID_ARG, "null argument");
    Layout L;
    int rc = make_layout(projs, n_projs, 1, max_rank, 1, &L);
    if (rc) return rc;
    return pack_adapter_slab(L, rank, A_host, B_host, static_cast<uint16_t*>(slab_host));
}

int bdlora_adapter_elems(const bdlora_proj_desc* projs, int32_t n_projs, int32_t rank, int64_t* elems) {
    if (!elems) return fail(BDLORA_ERR_INVALID_ARG, "null output");
    if (rank < 0) return fail(BDLORA_ERR_INVALID_ARG, "negative rank");
    Layout L;
    int rc = make_layout(projs, n_projs, 1, 0, 1, &L);
    if (rc) return rc;
    long long e = 0;
    for (int p = 0; p < n_projs; ++p)
        for (int s = 0; s < L.proj[p].S; ++s)
            e += (long long)L.proj[p].K * rank + (long long)rank * L.proj[p].slice_out[s];
    *elems = e;
    return BDLORA_OK;
}

int bdlora_pool_size(const bdlora_proj_desc* projs, int32_t n_projs, int32_t max_slots, int32_t max_rank,
                     int32_t max_tokens, int64_t* slab_bytes, int64_t* workspace_bytes) {
    Layout L;
    int rc = make_layout(projs, n_projs, max_slots, max_rank, max_tokens, &L);
    if (rc) return rc;
    if (slab_bytes) *slab_bytes = L.slab_bytes;
    if (workspace_bytes) *workspace_bytes = L.ws_bytes;
    return BDLORA_OK;
}

int bdlora_build_plan(const int32_t* loaded, int32_t max_slots, const int32_t* ids, int32_t T, int32_t* vid,
                      int32_t* gslot, int32_t* gstart, int32_t* gcount, int32_t* perm, int32_t* n_groups) {
    if (T < 0) return fail(BDLORA_ERR_INVALID_ARG, "negative T");
    if (max_slots < 1 || max_slots > BDLORA_MAX_SLOTS) return fail(BDLORA_ERR_INVALID_ARG, "bad max_slots");
    if (!loaded || !n_groups || (T > 0 && (!ids || !vid || !gslot || !gstart || !gcount || !perm)))
        return fail(BDLORA_ERR_INVALID_ARG, "null pointer");
    std::vector<int> cnt(max_slots, 0);
    bool bad = false;
    for (int t = 0; t < T; ++t) {
        const int a = ids[t];
        const bool ok = a >= 0 && a < max_slots && loaded[a] != 0;
        if (!ok && a != -1) bad = true;
        vid[t] = ok ? a : -1;
        if (ok) ++cnt[a];
    }
    int g = 0, off = 0;
    std::vector<int> cursor(max_slots, 0);
    for (int s = 0; s < max_slots; ++s) {
        cursor[s] = off;
        if (cnt[s] > 0) {
            gslot[g] = s;
            gstart[g] = off;
            gcount[g] = cnt[s];
            ++g;
        }
        off += cnt[s];
    }
    for (int t = 0; t < T; ++t)
        if (vid[t] >= 0) perm[cursor[vid[t]]++] = t;
    *n_groups = g;
    if (bad) return fail(BDLORA_ERR_BAD_ADAPTER, "an id names no loaded adapter slot");
    return BDLORA_OK;
}

int bdlora_create_pool(const bdlora_proj_desc* projs, int32_t n_projs, int32_t max_slots, int32_t max_rank,
                       int32_t max_tokens, int64_t pool_bytes, int32_t device, bdlora_pool_t* out) {
    if (!out) return fail(BDLORA_ERR_INVALID_ARG, "null output handle");
    *out = nullptr;
    if (pool_bytes < 0) return fail(BDLORA_ERR_INVALID_ARG, "pool_bytes must be >= 0");
    if (max_slots == 0 && pool_bytes > 0) {
        // as many slots as the adapter budget holds
        Layout L1;
        int rc = make_layout(projs, n_projs, 1, max_rank, max_tokens, &L1);
        if (rc) return rc;
        const long long per = L1.slot_stride * 2;
        const long long n = std::min<long long>(pool_bytes / per, BDLORA_MAX_SLOTS);
        if (n < 1)
            return fail(BDLORA_ERR_OOM, "pool_bytes " + std::to_string(pool_bytes) + " holds no adapter slot of " +
                                            std::to_string(per) + " bytes");
        max_slots = (int32_t)n;
    }
    Layout L;
    int rc = make_layout(projs, n_projs, max_slots, max_rank, max_tokens, &L);
    if (rc) return rc;
    if (pool_bytes > 0 && L.slab_bytes > pool_bytes)
        return fail(BDLORA_ERR_OOM, std::to_string(max_slots) + " adapter slots need " + std::to_string(L.slab_bytes) +
                                        " bytes, more than pool_bytes " + std::to_string(pool_bytes));
    int ndev = 0;
    if (hipGetDeviceCount(&ndev) != hipSuccess || ndev <= 0) {
        (void)hipGetLastError();
        return fail(BDLORA_ERR_UNSUPPORTED, "no HIP device");
    }
    if (device < 0 || device >= ndev) return fail(BDLORA_ERR_INVALID_ARG, "bad device index");
    hipDeviceProp_t prop;
    BDL_HIP(hipGetDeviceProperties(&prop, device));
    if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
        return fail(BDLORA_ERR_UNSUPPORTED, std::string("device is ") + prop.gcnArchName + ", need gfx950");
    DeviceGuard guard(device);
    if (!guard.ok) return fail(BDLORA_ERR_HIP, "hipSetDevice failed");

    bdlora_pool* P = new bdlora_pool();
    P->device = device;
    P->L = L;
    P->n_cu = std::max(1, prop.multiProcessorCount);
    long long tot = 0;
    const int S = max_slots, MT = max_tokens;
#define BDL_TRY(x)         \
    do {                   \
        int r_ = (x);      \
        if (r_) {          \
            free_pool(P);  \
            return r_;     \
        }                  \
    } while (0)
    BDL_TRY(dev_alloc(&P->d_slabs, (long long)S * L.slot_stride, &tot));
    BDL_TRY(dev_alloc(&P->d_r8, S, &tot));
    BDL_TRY(dev_alloc(&P->d_scale, S, &tot));
    BDL_TRY(dev_alloc(&P->d_loaded, S, &tot));
    BDL_TRY(dev_alloc(&P->d_vid, MT, &tot));
    BDL_TRY(dev_alloc(&P->d_tr8, MT, &tot));
    BDL_TRY(dev_alloc(&P->d_tgrp, MT, &tot));
    BDL_TRY(dev_alloc(&P->d_part, L.part_slots * bdl::kPartElems, &tot));
    BDL_TRY(dev_alloc(&P->d_mlp, L.mlp_elems, &tot));
    if (L.bigpart_elems > 0) BDL_TRY(dev_alloc(&P->d_bigpart, L.bigpart_elems, &tot));
    if (L.shrinkpart_elems > 0) BDL_TRY(dev_alloc(&P->d_shrinkpart, L.shrinkpart_elems, &tot));
    BDL_TRY(dev_alloc(&P->d_perm, MT, &tot));
    BDL_TRY(dev_alloc(&P->d_rowtok, MT, &tot));
    BDL_TRY(dev_alloc(&P->d_rowslot, MT, &tot));
    BDL_TRY(dev_alloc(&P->d_gslot, S + 1, &tot));
    BDL_TRY(dev_alloc(&P->d_gr8, bdl::kDecodeMaxT + 1, &tot));
    BDL_TRY(dev_alloc(&P->d_gstart, S + 1, &tot));
    BDL_TRY(dev_alloc(&P->d_gcount, S + 1, &tot));
    P->items_cap = (long long)S + MT / 16 + 2;
    BDL_TRY(dev_alloc(&P->d_items, P->items_cap, &tot));
    P->oct_elems = ((long long)MT / 16 + 1) * (16LL * L.r8max / 8 + 64);
    P->oct_elems = std::max(P->oct_elems, ((long long)MT / 64 + 1) * (64LL * L.r8max / 8 + 64));
    BDL_TRY(dev_alloc(&P->d_tile_oct, P->oct_elems, &tot));
    BDL_TRY(dev_alloc(&P->d_meta, 4, &tot));
    BDL_TRY(dev_alloc(&P->d_err, 1, &tot));
    long long stage = 0;
    for (int p = 0; p < n_projs; ++p) {
        BDL_TRY(dev_alloc(&P->d_Z[p], L.z_elems[p], &tot));
        BDL_TRY(dev_alloc(&P->d_Xp[p], L.xp_elems[p], &tot));
        const ProjInfo& pi = L.proj[p];
        stage = std::max(stage, (long long)pi.S * pi.K * std::max(1, max_rank) + (long long)std::max(1, max_rank) * pi.N);
    }
    BDL_TRY(dev_alloc(&P->d_stage, stage, &tot));
    P->stage_elems = stage;
    P->bytes = tot;
    auto hipz = [&](void* p, size_t n) -> int {
        hipError_t e = hipMemset(p, 0, n);
        if (e != hipSuccess) {
            free_pool(P);
            return fail(BDLORA_ERR_HIP, std::string("hipMemset: ") + hipGetErrorString(e));
        }
        return BDLORA_OK;
    };
    // zero everything the kernels may read: slabs (padding), tables, Z, flags
    if (int r = hipz(P->d_slabs, (size_t)S * L.slot_stride * 2)) return r;
    if (int r = hipz(P->d_r8, (size_t)S * 4)) return r;
    if (int r = hipz(P->d_scale, (size_t)S * 4)) return r;
    if (int r = hipz(P->d_loaded, (size_t)S * 4)) return r;
    if (int r = hipz(P->d_err, 4)) return r;
    if (int r = hipz(P->d_meta, 16)) return r;
    // plan tables: entries past a batch's counts are never written by the
    // plan; zero (slot 0) rather than whatever the allocation held
    if (int r = hipz(P->d_gslot, (size_t)(S + 1) * 4)) return r;
    if (int r = hipz(P->d_gr8, (size_t)(bdl::kDecodeMaxT + 1) * 4)) return r;
    if (int r = hipz(P->d_gstart, (size_t)(S + 1) * 4)) return r;
    if (int r = hipz(P->d_gcount, (size_t)(S + 1) * 4)) return r;
    for (int p = 0; p < n_projs; ++p)
        if (int r = hipz(P->d_Z[p], (size_t)std::max(1LL, L.z_elems[p]) * 2)) return r;
    hipError_t e = hipStreamCreateWithFlags(&P->load_stream, hipStreamNonBlocking);
    if (e == hipSuccess) e = hipStreamCreateWithFlags(&P->side_stream, hipStreamNonBlocking);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&P->fork_ev, hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&P->join_ev, hipEventDisableTiming);
    if (e != hipSuccess) {
        free_pool(P);
        return fail(BDLORA_ERR_HIP, std::string("hipStreamCreate: ") + hipGetErrorString(e));
    }
    e = hipDeviceSynchronize();
    if (e != hipSuccess) {
        free_pool(P);
        return fail(BDLORA_ERR_HIP, std::string("hipDeviceSynchronize: ") + hipGetErrorString(e));
    }
    // set-up of the allocation-free entry point on this device (its failure
    // only disables that entry point)
    P->static_err = bdl::static_scratch_init(device);
    if (P->static_err != hipSuccess) (void)hipGetLastError();
#undef BDL_TRY
    P->h_rank.assign(S, 0);
    P->h_r8.assign(S, 0);
    P->h_loaded.assign(S, 0);
    P->h_scale.assign(S, 0.f);
    *out = P;
    return BDLORA_OK;
}

int bdlora_destroy_pool(bdlora_pool_t P) {
    if (!P) return fail(BDLORA_ERR_INVALID_ARG, "null pool");
    DeviceGuard guard(P->device);
    (void)hipDeviceSynchronize();
    free_pool(P);
    return BDLORA_OK;
}

int bdlora_pool_slots(bdlora_pool_t P, int32_t* slots) {
    if (!P || !slots) return fail(BDLORA_ERR_INVALID_ARG, "null argument");
    *slots = P->L.max_slots;
    return BDLORA_OK;
}

int bdlora_pool_bytes(bdlora_pool_t P, int64_t* bytes) {
    if (!P || !bytes) return fail(BDLORA_ERR_INVALID_ARG, "null argument");
    *bytes = P->bytes;
    return BDLORA_OK;
}

static int upload_slot_tables(bdlora_pool_t P, int slot) {
    BDL_HIP(hipMemcpyAsync(P->d_r8 + slot, &P->h_r8[slot], 4, hipMemcpyHostToDevice, P->load_stream));
    BDL_HIP(hipMemcpyAsync(P->d_scale + slot, &P->h_scale[slot], 4, hipMemcpyHostToDevice, P->load_stream));
    BDL_HIP(hipMemcpyAsync(P->d_loaded + slot, &P->h_loaded[slot], 4, hipMemcpyHostToDevice, P->load_stream));
    BDL_HIP(hipStreamSynchronize(P->load_stream));
    return BDLORA_OK;
}

int bdlora_load_adapter(bdlora_pool_t P, int32_t slot, int32_t rank, float scale, const uint16_t* const* A_host,
                        const uint16_t* const* B_host) {
    if (!P) return fail(BDLORA_ERR_INVALID_ARG, "null pool");
    const Layout& L = P->L;
    if (slot < 0 || slot >= L.max_slots) return fail(BDLORA_ERR_INVALID_ARG, "slot out of range");
    if (rank < 0 || rank > L.max_rank) return fail(BDLORA_ERR_INVALID_ARG, "rank out of range 0..max_rank");
    if (!std::isfinite(scale)) return fail(BDLORA_ERR_INVALID_ARG, "scale must be finite");
    if (rank > 0 && (!A_host || !B_host)) return fail(BDLORA_ERR_INVALID_ARG, "null factor arrays");
    const int r8 = rank8(rank);
    // host-side checks first: every factor present and finite
    int k = 0;
    for (int p = 0; p < L.n_projs; ++p) {
        const ProjInfo& pi = L.proj[p];
        for (int s = 0; s < pi.S; ++s, ++k) {
            if (rank == 0) continue;
            const uint16_t* a = A_host[k];
            const uint16_t* b = B_host[k];
            if (!a || !b) return fail(BDLORA_ERR_INVALID_ARG, "null factor pointer");
            const long long na = (long long)pi.K * rank, nb = (long long)rank * pi.slice_out[s];
            for (long long i = 0; i < na; ++i)
                if ((a[i] & 0x7f80u) == 0x7f80u) return fail(BDLORA_ERR_INVALID_ARG, "non-finite value in A");
            for (long long i = 0; i < nb; ++i)
                if ((b[i] & 0x7f80u) == 0x7f80u) return fail(BDLORA_ERR_INVALID_ARG, "non-finite value in B");
        }
    }
    DeviceGuard guard(P->device);
    if (!guard.ok) return fail(BDLORA_ERR_HIP, "hipSetDevice failed");
    // mark the slot empty while it is rewritten
    P->h_loaded[slot] = 0;
    if (int rc = upload_slot_tables(P, slot)) return rc;
    k = 0;
    for (int p = 0; p < L.n_projs; ++p) {
        const ProjInfo& pi = L.proj[p];
        uint16_t* slab = P->d_slabs + (long long)slot * L.slot_stride;
        if (rank > 0) {
            long long off = 0;
            for (int s = 0; s < pi.S; ++s) {
                const long long n = (long long)pi.K * rank;
                BDL_HIP(hipMemcpyAsync(P->d_stage + off, A_host[k + s], n * 2, hipMemcpyHostToDevice, P->load_stream));
                off += n;
            }
            for (int s = 0; s < pi.S; ++s) {
                const long long n = (long long)rank * pi.slice_out[s];
                BDL_HIP(hipMemcpyAsync(P->d_stage + off, B_host[k + s], n * 2, hipMemcpyHostToDevice, P->load_stream));
                off += n;
            }
            BDL_HIP(bdl::launch_pack_adapter(slab + pi.a_off, slab + pi.b_off, P->d_stage, pi.K, pi.S,
                                             pi.slice_out, rank, r8, P->load_stream));
            BDL_HIP(hipStreamSynchronize(P->load_stream));   // stage is reused by the next projection
        }
        k += pi.S;
    }
    P->h_rank[slot] = rank;
    P->h_r8[slot] = r8;
    P->h_scale[slot] = scale;
    P->h_loaded[slot] = 1;
    return upload_slot_tables(P, slot);
}

int64_t bdlora_slot_bytes(bdlora_pool_t P) {
    return P ? P->L.slot_stride * 2 : 0;
}

int bdlora_pack_adapter_host(bdlora_pool_t P, int32_t rank, const uint16_t* const* A_host,
                             const uint16_t* const* B_host, void* slab_host) {
    if (!P || !slab_host) return fail(BDLORA_ERR_INVALID_ARG, "null argument");
    return pack_adapter_slab(P->L, rank, A_host, B_host, static_cast<uint16_t*>(slab_host));
}

int bdlora_load_adapters_packed(bdlora_pool_t P, int32_t first_slot, int32_t n, const int32_t* ranks,
                                const float* scales, const void* slabs_host, void* stream) {
    if (!P || !slabs_host || !ranks || !scales) return fail(BDLORA_ERR_INVALID_ARG, "null argument");
    const Layout& L = P->L;
    if (n < 1 || n > bdl::kMaxSlotBatch) return fail(BDLORA_ERR_INVALID_ARG, "n must be 1..64");
    if (first_slot < 0 || first_slot + n > L.max_slots) return fail(BDLORA_ERR_INVALID_ARG, "slots out of range");
    bdl::SlotBatch sb;
    sb.first = first_slot;
    sb.n = n;
    for (int i = 0; i < n; ++i) {
        if (ranks[i] < 0 || ranks[i] > L.max_rank) return fail(BDLORA_ERR_INVALID_ARG, "rank out of range 0..max_rank");
        if (!std::isfinite(scales[i])) return fail(BDLORA_ERR_INVALID_ARG, "scale must be finite");
        sb.r8[i] = rank8(ranks[i]);
        sb.scale[i] = scales[i];
    }
    DeviceGuard guard(P->device);
    if (!guard.ok) return fail(BDLORA_ERR_HIP, "hipSetDevice failed");
    hipStream_t s = (hipStream_t)stream;
    // consecutive slots are one contiguous range of the pool: one copy
    BDL_HIP(hipMemcpyAsync(P->d_slabs + (long long)first_slot * L.slot_stride, slabs_host,
                           (size_t)n * L.slot_stride * 2, hipMemcpyHostToDevice, s));
    BDL_HIP(bdl::launch_set_slots(P->d_r8, P->d_scale, P->d_loaded, sb, s));
    for (int i = 0; i < n; ++i) {
        P->h_rank[first_slot + i] = ranks[i];
        P->h_r8[first_slot + i] = sb.r8[i];
        P->h_scale[first_slot + i] = scales[i];
        P->h_loaded[first_slot + i] = 1;
    }
    return BDLORA_OK;
}

int bdlora_load_adapter_packed(bdlora_pool_t P, int32_t slot, int32_t rank, float scale, const void* slab_host,
                               void* stream) {
    return bdlora_load_adapters_packed(P, slot, 1, &rank, &scale, slab_host, stream);
}

int bdlora_unload_adapter(bdlora_pool_t P, int32_t slot) {
    if (!P) return fail(BDLORA_ERR_INVALID_ARG, "null pool");
    if (slot < 0 || slot >= P->L.max_slots) return fail(BDLORA_ERR_INVALID_ARG, "slot out of range");
    DeviceGuard guard(P->device);
    if (!guard.ok) return fail(BDLORA_ERR_HIP, "hipSetDevice failed");
    P->h_loaded[slot] = 0;
    P->h_rank[slot] = 0;
    P->h_r8[slot] = 0;
    return upload_slot_tables(P, slot);
}

// Kernel shapes by batch size: decode batches use short row tiles and narrow
// shrink items (more workgroups), prefill batches the largest tiles.
struct Shapes {
    int smb, snb;   // shrink row / column blocks of 16
    int gmb, gnb;   // base GEMM row / column blocks of 16
};

// Column blocks per base-GEMM tile: the widest tile (least re-reading of the
// activations) that still leaves enough workgroups to occupy the chip.
static Shapes pick_shapes(int T, long long col_blocks = 0, int r8max = bdl::kMaxRank8) {
    Shapes k;
    // prefill shrink items: 64 rows x 64 rank columns; when no adapter is
    // wider than rank 32, 32 rows x 96 columns, so that the three slices of
    // a q/k/v projection come out of one pass over its rows of X
    k.smb = T <= 512 ? 1 : (r8max <= 32 ? 2 : 4);
    k.snb = T <= 512 ? 1 : (r8max <= 32 ? 6 : 4);
    k.gmb = T <= 16 ? 1 : (T <= 32 ? 2 : 4);
    const long long row_tiles = (T + 16 * k.gmb - 1) / (16 * k.gmb);
    const long long blocks = col_blocks * row_tiles;
    k.gnb = blocks >= 4 * 192 ? 4 : (blocks >= 2 * 192 ? 2 : 1);
    return k;
}

static int oct_cap(const Layout& L, int gemm_mt) { return gemm_mt * L.r8max / 8 + 64; }

static void fill_plan_args(bdlora_pool_t P, const Batch& B, int T, bdl::PrepArgs* a, const Shapes& k) {
    a->ids = B.ids;
    a->T = T;
    a->n_seg = B.ids ? 0 : B.n_seg;
    for (int i = 0; i < a->n_seg; ++i) {
        a->seg_start[i] = B.seg_start[i];
        a->seg_slot[i] = B.seg_slot[i];
    }
    a->act_max = -1;
    a->loaded = P->d_loaded;
    a->r8 = P->d_r8;
    a->max_slots = P->L.max_slots;
    a->mts = 16 * k.smb;
    a->gemm_mt = 16 * k.gmb;
    a->oct_cap = oct_cap(P->L, 16 * k.gmb);
    a->vid = P->d_vid;
    a->tr8 = P->d_tr8;
    a->tgrp = nullptr;
    a->perm = P->d_perm;
    a->rowtok = nullptr;
    a->rowslot = nullptr;
    a->oct_perm = 0;
    a->gslot = P->d_gslot;
    a->gr8 = nullptr;
    a->gstart = P->d_gstart;
    a->gcount = P->d_gcount;
    a->items = P->d_items;
    a->tile_oct = P->d_tile_oct;
    a->meta = P->d_meta;
    a->err = P->d_err;
    a->n_jobs = 0;
    a->total_frags = 0;
    a->decode_plan = 0;
}

// Decode batches: prep (plan + activation packing), the split-K main launch
// over W_s and the used adapters' A^T, the epilogue.
// How a call uses the decode launches: the MLP chains two calls, the second
// reusing the first's plan and reading the intermediate the first's epilogue
// packed.
struct DecMode {
    bool prep = true;              // plan the batch and pack the activations (false: the tables hold this
                                   // batch's plan and Xp its activations); at most 16 tokens the main
                                   // launch plans it and reads the caller's X, with no prep launch
    int mlp_act = -1;              // >= 0: the epilogue writes the MLP intermediate
    uint16_t* h_dst = nullptr;     // where (fragment layout of the second projection's input)
    int h_KS = 0;
};

// scales of a packed INT4 base weight (null for a bf16 base)
static const uint16_t* int4_scales(const ProjInfo& pi, const void* W) {
    if (pi.wfmt != BDLORA_WEIGHT_INT4_G128) return nullptr;
    return reinterpret_cast<const uint16_t*>(static_cast<const char*>(W) + (size_t)pi.N * pi.K / 2);
}

// Where a decode call keeps its per-batch scratch: the pool's workspace, or
// (the allocation-free entry point) the library's static device array.
struct DecWs {
    int* vid = nullptr;               // [T] validated ids
    int* tr8 = nullptr;               // [T] padded rank of each token's adapter
    int* tgrp = nullptr;              // [T] group of each token's adapter
    int* gslot = nullptr;             // [<= 64] slots of the adapters in use
    int* gr8 = nullptr;               // [<= 64] their padded ranks
    int* meta = nullptr;              // [4] plan counts
    uint16_t* Xp[bdl::kMaxProjs] = {};   // packed activations of the call's i-th projection
    float* part = nullptr;            // fp32 partial tiles; null: carved from arena
    long long part_slots = 0;
    char* arena = nullptr;            // static scratch left for the partial tiles
    long long arena_bytes = 0;
};

static DecWs pool_dec_ws(bdlora_pool_t P, int n, const int32_t* projs) {
    DecWs w;
    w.vid = P->d_vid;
    w.tr8 = P->d_tr8;
    w.tgrp = P->d_tgrp;
    w.gslot = P->d_gslot;
    w.gr8 = P->d_gr8;
    w.meta = P->d_meta;
    for (int i = 0; i < n; ++i) w.Xp[i] = P->d_Xp[projs[i]];
    w.part = P->d_part;
    w.part_slots = P->L.part_slots;
    return w;
}

static int forward_decode(bdlora_pool_t P, int n, const int32_t* projs, const void* const* X,
                          const void* const* W, void* const* out, const Batch& B, int T, hipStream_t s,
                          const DecWs& ws, const DecMode& mode = DecMode()) {
    const Layout& L = P->L;
    // small batches: the main launch plans the batch in every wave and
    // gathers the caller's X, so no prep launch runs.  The gathered rows
    // slow the main launch with the activation bytes (measured: a 17..32
    // token batch of the 70B layer shard, 58 KB of activations per token,
    // gains up to about 28 tokens, the 8B shard, 29 KB per token, at every
    // size up to 32; at 64 tokens the prep launch is cheaper)
    static_assert(BDLORA_DECODE_PLAN_IN_MAIN_T <= 32, "the planning kernel takes at most two row blocks");
    long long act_bytes = 0;
    for (int i = 0; i < n; ++i) act_bytes += 2LL * T * L.proj[projs[i]].K;
    const bool fold = mode.prep && (T <= 16 || (T <= BDLORA_DECODE_PLAN_IN_MAIN_T &&
                                                act_bytes <= BDLORA_DECODE_PLAN_IN_MAIN_BYTES));
    // adapter positions of the launches: the loaded adapters bound the
    // distinct ones a batch can use (the plan treats any past that bound as
    // none and raises the error flag).  Both forms of the batch (ids,
    // segments) take the same launch geometry, so they give the same bits.
    int n_loaded = 0;
    for (int v : P->h_loaded) n_loaded += v != 0;
    const int act_max = std::min({T, n_loaded, bdl::kDecodeMaxT});

    bdl::DecArgs da;
    std::memset(&da, 0, sizeof(da));
    long long units_min = 0, units_max = 0, groups_max = 0;
    int tiles = 0;
    for (int i = 0; i < n; ++i) {
        const ProjInfo& pi = L.proj[projs[i]];
        bdl::DecProj& d = da.p[i];
        d.X = fold ? (const uint16_t*)X[i] : nullptr;
        d.Xp = ws.Xp[i];
        d.W = (const uint16_t*)W[i];
        d.Ws = int4_scales(pi, W[i]);
        d.out = (uint16_t*)out[i];
        d.K = pi.K;
        d.N = pi.N;
        d.n_slices = pi.S;
        for (int t = 0; t <= bdl::kMaxSlices; ++t) d.slice_col[t] = pi.slice_col[t];
        d.a_off = pi.a_off;
        d.b_off = pi.b_off;
        d.nWb = pi.N / 16;
        d.nbA = (pi.S * L.r8max + 15) / 16;
        d.tile_base = tiles;
        tiles += (pi.N + 63) / 64;
        units_min += (long long)d.nWb * (pi.K / 32);
        units_max += (d.nWb + (long long)act_max * d.nbA) * (pi.K / 32);
        groups_max += (d.nWb + (long long)act_max * d.nbA + 3) / 4;
    }
    // two workgroups per CU, each with at least 64 units (16 k-steps of a
    // full group) whatever the number of adapters in use; fewer, longer
    // workgroups split each output group over fewer partial tiles, which its
    // epilogue adds one by one.  Measured with the data streamed from HBM: a
    // layer whose base weights give one to two such workgroups per CU is
    // fastest on one per CU of at least 128 units (the 8B MLP's gate and up
    // at 64 tokens, 448 64-unit workgroups: 54.1 -> 51.1 us a step); a
    // smaller one keeps 64-unit workgroups (one 1792-column projection at 16
    // tokens: 20.7 -> 17.5 us from two per CU, 18.1 with 128-unit ones); a
    // larger one two per CU (the 8B decode layer, 832 64-unit workgroups).
    // The kernels' 32-bit schedule arithmetic needs units * workgroups < 2^32
    // (at least one workgroup: one that owns every unit needs no minimum)
    const long long min_units = units_min >= 64LL * P->n_cu && units_min < 64LL * 2 * P->n_cu ? 128 : 64;
    const int grid = (int)std::min<long long>(
        {2LL * P->n_cu, (long long)bdl::kDecMaxGrid, std::max(1LL, units_min / min_units),
         0xffffffffLL / std::max(1LL, units_max)});
    if (grid < 1) return fail(BDLORA_ERR_SHAPE, "batch too large for the decode launch's schedule");
    float* part = ws.part;
    long long part_slots = ws.part_slots;
    if (!part) {
        // the partial tiles this call needs, from the rest of the static scratch
        part_slots = groups_max + grid;
        if (part_slots * bdl::kPartElems * 4 > ws.arena_bytes)
            return fail(BDLORA_ERR_SHAPE, "the call's partial tiles need " +
                                              std::to_string(part_slots * bdl::kPartElems * 4) +
                                              " bytes, the static scratch has " + std::to_string(ws.arena_bytes) +
                                              " left after the plan and the packed activations");
        part = reinterpret_cast<float*>(ws.arena);
    }
    if (groups_max + grid > part_slots) return fail(BDLORA_ERR_SHAPE, "batch exceeds the pool workspace");
    da.n_proj = n;
    da.T = T;
    {
        unsigned u = 0;
        int g = 0;
        for (int i = 0; i < n; ++i) {
            const int nb = da.p[i].nWb + act_max * da.p[i].nbA;
            da.sub[i] = u;
            da.sgb[i] = g;
            da.snb[i] = nb;
            da.sks[i] = da.p[i].K / 32;
            da.stb[i] = da.p[i].tile_base;
            u += (unsigned)nb * (unsigned)da.sks[i];
            g += (nb + 3) / 4;
        }
        da.units = u;
    }
    da.pool = P->d_slabs;
    da.slot_stride = L.slot_stride;
    da.scale = P->d_scale;
    da.vid = ws.vid;
    da.tr8 = ws.tr8;
    da.tgrp = ws.tgrp;
    da.gslot = ws.gslot;
    da.gr8 = ws.gr8;
    da.meta = ws.meta;
    da.act_max = act_max;
    da.part = part;
    da.part_slots = (int)part_slots;
    da.main_grid = grid;
    da.tiles = tiles;
    da.err = P->d_err;
    da.mlp_act = mode.mlp_act;
    da.h_dst = mode.h_dst;
    da.h_KS = mode.h_KS;

    Shapes k;
    k.smb = 1;
    k.snb = 4;
    k.gmb = (T + 15) / 16;
    k.gnb = 4;
    bdl::PrepArgs pa;
    fill_plan_args(P, B, T, &pa, k);
    pa.tile_oct = nullptr;                        // the epilogue needs no octet lists
    pa.decode_plan = 1;                           // writes vid, tr8, tgrp, gslot, meta (and err) only
    pa.vid = ws.vid;
    pa.tr8 = ws.tr8;
    pa.tgrp = ws.tgrp;
    pa.gslot = ws.gslot;
    pa.gr8 = ws.gr8;
    pa.meta = ws.meta;
    pa.perm = nullptr;
    pa.gstart = pa.gcount = nullptr;
    pa.items = nullptr;
    pa.act_max = act_max;
    // projections given the same X (gate and up) share one packed copy
    int frags = 0, jobs = 0;
    for (int q = 0; q < n && mode.prep; ++q) {
        int same = -1;
        for (int r = 0; r < q && same < 0; ++r)
            if (X[r] == X[q] && da.p[r].K == da.p[q].K) same = r;
        if (same >= 0) {
            da.p[q].Xp = da.p[same].Xp;
            continue;
        }
        bdl::PackJob& J = pa.jobs[jobs++];
        J.src = (const uint16_t*)X[q];
        J.dst = ws.Xp[q];
        J.rows = T;
        J.K = da.p[q].K;
        J.frag_base = frags;
        frags += ((T + 15) / 16) * (J.K / 32);
    }
    pa.n_jobs = jobs;
    pa.total_frags = frags;

    hipEvent_t* ev = nullptr;
    if (P->prof_left > 0 && (size_t)(P->prof_used + 1) * kProfEvents <= P->prof_ev.size()) {
        ev = &P->prof_ev[(size_t)P->prof_used * kProfEvents];
        ++P->prof_used;
        --P->prof_left;
    }
    if (fold) {
        // the plan's inputs for the main launch
        da.plan = 1;
        da.ids = B.ids;
        da.n_seg = B.ids ? 0 : B.n_seg;
        if (da.n_seg > bdl::kDecodeMaxT) return fail(BDLORA_ERR_INVALID_ARG, "more segments than tokens");
        for (int i = 0; i < da.n_seg; ++i) {
            da.seg_start[i] = B.seg_start[i];
            da.seg_slot[i] = B.seg_slot[i];
        }
        da.loaded = P->d_loaded;
        da.r8 = P->d_r8;
        da.max_slots = L.max_slots;
    }
    if (ev) BDL_HIP(hipEventRecord(ev[0], s));
    if (mode.prep && !fold) BDL_HIP(bdl::launch_prep(pa, s));
    if (ev) BDL_HIP(hipEventRecord(ev[1], s));
    if (ev) BDL_HIP(hipEventRecord(ev[2], s));
    BDL_HIP(bdl::launch_dec_main(da, k.gmb, s));
    if (ev) BDL_HIP(hipEventRecord(ev[3], s));
    if (ev) BDL_HIP(hipEventRecord(ev[4], s));
    BDL_HIP(bdl::launch_dec_epi(da, s));
    if (ev) BDL_HIP(hipEventRecord(ev[5], s));
    if (ev) BDL_HIP(hipEventRecord(ev[6], s));
    if (ev) BDL_HIP(hipEventRecord(ev[7], s));
    P->last_path = BDLORA_PATH_DECODE;
    return BDLORA_OK;
}

static bool use_decode(const Layout& L, int T) {
    // the decode launches address their partial tiles with 32-bit byte offsets
    return T <= bdl::kDecodeMaxT && L.part_slots * bdl::kPartElems * 4 < (1LL << 31);
}

// Batches above the decode size: prep (plan + packing; with pack = false the
// packed activations are already in place), shrink, base product with the
// expand fused in.
// The MLP's first projections (bdlora_forward_mlp, batches above the decode
// size): where H goes and how it is formed.
struct MlpOut {
    int act;                 // BDLORA_ACT_*
    uint16_t* h;             // H in the fragment layout of down's input
    int h_KS;                // its k-steps (down's d_in / 32)
    float* f32[2];           // 64-row path: the projections' fp32 outputs (formed into H afterwards)
};

static int forward_prefill(bdlora_pool_t P, int n, const int32_t* projs, const void* const* X,
                           const void* const* W, void* const* out, const Batch& B, int T, hipStream_t s,
                           bool pack = true, const MlpOut* mlp = nullptr) {
    const Layout& L = P->L;
    long long col_blocks = 0;
    for (int i = 0; i < n; ++i) col_blocks += L.proj[projs[i]].N / 16;
    const Shapes k = pick_shapes(T, col_blocks, L.r8max);
    const int mts = 16 * k.smb, nts = 16 * k.snb;
    const int MT = 16 * k.gmb, NT = 16 * k.gnb;

    bdl::FwdArgs fa;
    std::memset(&fa, 0, sizeof(fa));
    // heavy projections first so the long-running tiles start early
    std::vector<int> order(n);
    for (int i = 0; i < n; ++i) order[i] = i;
    if (!mlp)        // (the MLP's gate stays first: it leads the paired tiles)
        std::stable_sort(order.begin(), order.end(), [&](int x, int y) {
            return (long long)L.proj[projs[x]].K * L.proj[projs[x]].N >
                   (long long)L.proj[projs[y]].K * L.proj[projs[y]].N;
        });
    // the loaded adapters bound the distinct ones the batch can use; the
    // path choices below take that bound (the host does not see device ids,
    // and both forms of the batch must take the same launches)
    int n_loaded = 0;
    for (int v : P->h_loaded) n_loaded += v != 0;
    // bf16 weights above one 256-row tile: the 256 x 256 LDS-staged kernel
    // (its octet lists are those of 64-row blocks, as planned for T > 32),
    // with long-K tiles split into k-ranges when the batch has too few tiles
    // to occupy the chip.  Batches of one row tile stay on the 64-row kernel:
    // they are weight-streaming bound, and the large tile streams its weight
    // through LDS at under half the rate that kernel reaches.
    bool big = T > bdl::kBigM && MT == 64 && P->d_bigpart != nullptr;
    for (int i = 0; i < n; ++i) {
        // its buffer loads take 32-bit byte offsets into the packed X and W
        const ProjInfo& pi = L.proj[projs[i]];
        const long long xb = ((long long)T + 15) / 16 * 16 * pi.K * 2, wb = (long long)pi.N * pi.K * 2;
        big = big && pi.wfmt == BDLORA_WEIGHT_BF16 && xb < (1LL << 31) && wb < (1LL << 31);
    }
    // bf16 weights at medium batches: all rows in one tile of the medium-batch
    // launch (each weight fragment read once), whose partials the 64-row
    // kernel adds to the expand.  8 waves x mid_nb column blocks per tile;
    // long-K tiles are cut into k-ranges of about q k-steps so that the
    // items fill the chip once, every item storing one partial tile.
    bool mid = !big && T > bdl::kDecodeMaxT && T <= bdl::kMidMaxT && MT == 64 && P->d_bigpart != nullptr;
    for (int i = 0; i < n; ++i) {
        const ProjInfo& pi = L.proj[projs[i]];
        const long long xb = ((long long)T + 15) / 16 * 16 * pi.K * 2, wb = (long long)pi.N * pi.K * 2;
        mid = mid && pi.wfmt == BDLORA_WEIGHT_BF16 && xb < (1LL << 31) && wb < (1LL << 31);
    }
    const int mid_nb = 2, mid_rb = T <= 128 ? 8 : 16, mid_tn = 128 * mid_nb;
    int mid_split[bdl::kMaxProjs];
    int mid_items = 0;
    if (mid) {
        long long work = 0;
        for (int i = 0; i < n; ++i) {
            const ProjInfo& pi = L.proj[projs[i]];
            work += (long long)((pi.N + mid_tn - 1) / mid_tn) * (pi.K / 32);
        }
        const long long units = std::min<long long>(P->n_cu, bdl::kBigPartSlots);
        for (long long q = std::max(1LL, (work + units - 1) / units);; ++q) {
            mid_items = 0;
            for (int i = 0; i < n; ++i) {
                const ProjInfo& pi = L.proj[projs[i]];
                mid_split[i] = (int)std::max(1LL, (long long)(pi.K / 32) / q);
                mid_items += (pi.N + mid_tn - 1) / mid_tn * mid_split[i];
            }
            if (mid_items <= bdl::kBigPartSlots) break;
            // every tile unsplit and still more partials than the workspace holds
            if (q >= 1024) {
                mid = false;
                break;
            }
        }
        // The partials' round trip (written, then read by the epilogue) must
        // stay well below the weight bytes the launch saves re-reading: short
        // K ranges (small layers) make the partials as large as the weight,
        // and then the 64-row kernel is as fast or faster -- unless the batch
        // spreads over many adapters (at most 8 tokens per loaded adapter):
        // its shrink is then long, and this path runs it beside the base
        // product instead of before it.
        long long part_bytes = 0, w_bytes = 0;
        for (int i = 0; i < n; ++i) {
            const ProjInfo& pi = L.proj[projs[i]];
            part_bytes += (long long)((pi.N + mid_tn - 1) / mid_tn) * mid_split[i] * ((T + 15) / 16 * 16) * mid_tn * 4;
            w_bytes += (long long)pi.N * pi.K * 2;
        }
        mid = mid && (2 * part_bytes * 10 <= 6 * w_bytes || T <= 8 * n_loaded);
    }
    // MLP on the large-tile and medium-batch paths: their epilogues form H
    // and write it once, in bf16 (gate and up in paired tiles); on the
    // 64-row path the projections write fp32 and a pack launch forms H
    const bool h_fused = mlp && (big || mid);
    const bool paired = h_fused && mlp->act == BDLORA_ACT_SILU_MUL;
    const int tiles_m = (T + MT - 1) / MT;
    const int tm = big ? (T + bdl::kBigM - 1) / bdl::kBigM : tiles_m;
    const int tn = big ? (paired ? bdl::kBigN / 2 : bdl::kBigN) : NT;
    // Large tiles: a projection's tiles are cut into ksplit k-ranges of about
    // q k-steps, q = (all tile k-steps) / (compute units), so that the work
    // items fill the chip once; ksplit = 1 when its K is at most q.  The
    // split items' partials fit kBigPartSlots (sum of tiles x ksplit over the
    // split projections <= all tile k-steps / q <= the compute units used).
    int ksplit[bdl::kMaxProjs];
    for (int i = 0; i < n; ++i) ksplit[i] = 1;
    if (big) {
        long long work = 0;
        for (int i = 0; i < (paired ? 1 : n); ++i) {        // paired: the gate's tiles carry up's columns
            const ProjInfo& pi = L.proj[projs[i]];
            work += (long long)tm * ((pi.N + tn - 1) / tn) * (pi.K / 32);
        }
        const long long units = std::min<long long>(P->n_cu, bdl::kBigPartSlots);
        const long long q = std::max(1LL, (work + units - 1) / units);
        for (int i = 0; i < n; ++i) ksplit[i] = (int)std::max(1LL, (long long)(L.proj[projs[i]].K / 32) / q);
    }
    // row-major X (the caller's, on the large-tile path): its copies take the
    // two k-steps of a pair at once, so K must hold whole pairs and every
    // k-range at least one pair
    bool xrm = big && pack;
    for (int i = 0; i < n; ++i) xrm = xrm && L.proj[projs[i]].K % 64 == 0;
    if (xrm)
        for (int i = 0; i < n; ++i) ksplit[i] = std::min(ksplit[i], std::max(1, L.proj[projs[i]].K / 64));
    // the medium-batch GEMM's copies (one k-step of a row at a time) and its
    // shrink read the caller's X too, for any K
    if (mid && pack) xrm = true;
    int tile = 0, cch = 1, fix = 0, pslot = 0, mid_cols = 0;
    for (int q = 0; q < n; ++q) {
        const int i = order[q];
        const ProjInfo& pi = L.proj[projs[i]];
        bdl::ProjLaunch& pl = fa.p[q];
        pl.X = (const uint16_t*)X[i];
        pl.Xp = P->d_Xp[projs[i]];
        // the large and medium-batch tiles and their shrink gather rows of
        // the caller's X directly (32-bit offsets: T K 2 < 2^31 is part of
        // the paths' conditions); an intermediate already packed (pack
        // false) is read from Xp
        pl.x_rowmajor = xrm ? 1 : 0;
        pl.W = (const uint16_t*)W[i];
        pl.Ws = int4_scales(pi, W[i]);
        pl.out = (uint16_t*)out[i];
        pl.out_f32 = mlp && !h_fused ? mlp->f32[i] : nullptr;
        pl.Z = P->d_Z[projs[i]];
        pl.zplane = (long long)L.max_tokens * pi.zs;
        pl.K = pi.K;
        pl.N = pi.N;
        pl.n_slices = pi.S;
        pl.zs = pi.zs;
        for (int s = 0; s <= bdl::kMaxSlices; ++s) pl.slice_col[s] = pi.slice_col[s];
        pl.a_off = pi.a_off;
        pl.b_off = pi.b_off;
        pl.tiles_n = (pi.N + tn - 1) / tn;
        pl.tile_base = tile;
        pl.ksplit = ksplit[i];
        pl.fix_base = fix;
        pl.part_base = pslot;
        if (paired && q == 1) {
            // up has no tiles of its own (gate's tiles hold its columns): its
            // bases sit past every item so that none maps to it
            pl.ksplit = ksplit[0];
            pl.fix_count = 0;
        } else {
            tile += tm * pl.tiles_n * pl.ksplit;
            pl.fix_count = pl.ksplit > 1 ? tm * pl.tiles_n : 0;
            fix += pl.fix_count;
            pslot += pl.fix_count * pl.ksplit;
        }
        if (mid) {
            pl.ksplit = mid_split[i];
            pl.part_base = pslot;
            pslot += (pi.N + mid_tn - 1) / mid_tn * mid_split[i];
            pl.col_base = mid_cols;
            if (!(paired && q == 1)) mid_cols += (pi.N + 63) / 64;
        }
        cch = std::max(cch, (pi.S * L.r8max + nts - 1) / nts);
    }
    fa.n_proj = n;
    fa.T = T;
    fa.pool = P->d_slabs;
    fa.slot_stride = L.slot_stride;
    fa.r8max = L.r8max;
    fa.scale = P->d_scale;
    fa.vid = P->d_vid;
    fa.perm = P->d_perm;
    fa.items = P->d_items;
    fa.meta = P->d_meta;
    // every group gives at most ceil(count / mts) items: at most
    // (groups + T / mts) in all, groups bounded by the slots (device ids: a
    // bound that holds whatever is loaded when a captured forward replays)
    fa.items_bound = std::min(T, L.max_slots) + (T + mts - 1) / mts;
    fa.cchunks = cch;
    // Small batches over many adapters (groups of a few scattered tokens, at
    // most 8 per loaded adapter on average) split each shrink item's K over
    // the XCDs, partials in their own workspace.  Few large groups read X
    // about once anyway; there the split would only add the partials'
    // traffic.
    fa.shrink_kp = 1;
    fa.shrinkpart = P->d_shrinkpart;
    // the unsplit shrink's unit order: longest K first (its units' length),
    // so the short ones fill the end
    fa.queue = P->d_meta + 2;
    for (int q = 0; q < n; ++q) fa.sorder[q] = q;
    std::stable_sort(fa.sorder, fa.sorder + n, [&](int x, int y) { return fa.p[x].K > fa.p[y].K; });
    if (T <= 512 && T <= 8 * n_loaded && P->d_shrinkpart &&
        (long long)n * fa.items_bound * cch * bdl::kShrinkKP * mts * nts <= L.shrinkpart_elems)
        fa.shrink_kp = bdl::kShrinkKP;
    fa.tile_oct = P->d_tile_oct;
    fa.oct_cap = oct_cap(L, MT);
    fa.tiles_m = tm;
    fa.total_tiles = tile;
    fa.bigpart = P->d_bigpart;
    fa.fixup = 0;
    fa.total_fix = fix;
    fa.mid_rb = mid_rb;
    fa.mid_nb = mid_nb;
    fa.mid_items = mid ? mid_items : 0;
    fa.mid_col_tiles = mid ? mid_cols : 0;
    fa.max_slots = L.max_slots;
    fa.mlp_act = h_fused ? mlp->act : -1;
    fa.h_dst = h_fused ? mlp->h : nullptr;
    fa.h_KS = h_fused ? mlp->h_KS : 0;
    if (paired) {
        // up's bases past gate's items (and past the epilogue's column tiles)
        fa.p[1].tile_base = tile;
        fa.p[1].fix_base = fix;
        fa.p[1].col_base = mid_cols;
    }
    if (pslot > bdl::kBigPartSlots) return fail(BDLORA_ERR_SHAPE, "large-tile split exceeds its partial workspace");
    if (fa.items_bound > P->items_cap || (long long)tiles_m * fa.oct_cap > P->oct_elems)
        return fail(BDLORA_ERR_SHAPE, "batch exceeds the pool workspace");

    bdl::PrepArgs pa;
    fill_plan_args(P, B, T, &pa, k);
    if (big) {
        // the large tiles take their rows in adapter order
        pa.rowtok = P->d_rowtok;
        pa.oct_perm = 1;
        fa.rowtok = P->d_rowtok;
    } else if (mid) {
        // so do the medium-batch tiles (their expand needs no octet lists,
        // only each row's slot and rank)
        pa.rowtok = P->d_rowtok;
        pa.rowslot = P->d_rowslot;
        pa.tile_oct = nullptr;
        fa.rowtok = P->d_rowtok;
        fa.rowslot = P->d_rowslot;
    }
    int frags = 0, jobs = 0;
    for (int q = 0; q < n && pack; ++q) {
        if (fa.p[q].x_rowmajor) continue;
        bdl::PackJob& J = pa.jobs[jobs++];
        J.src = fa.p[q].X;
        J.dst = P->d_Xp[projs[order[q]]];
        J.rows = T;
        J.K = fa.p[q].K;
        J.frag_base = frags;
        frags += ((T + 15) / 16) * (J.K / 32);
    }
    pa.n_jobs = jobs;
    pa.total_frags = frags;

    hipEvent_t* ev = nullptr;
    if (P->prof_left > 0 && (size_t)(P->prof_used + 1) * kProfEvents <= P->prof_ev.size()) {
        ev = &P->prof_ev[(size_t)P->prof_used * kProfEvents];
        ++P->prof_used;
        --P->prof_left;
    }
    if (ev) BDL_HIP(hipEventRecord(ev[0], s));
    BDL_HIP(bdl::launch_prep(pa, s));
    if (ev) BDL_HIP(hipEventRecord(ev[1], s));
    // Medium batches: the shrink (Z for the epilogue) and the base product
    // are independent, and both stream HBM; the shrink runs on the pool's
    // side stream beside the base product and is joined back before the
    // epilogue.  The base product is enqueued first, so that its workgroups
    // (one per CU) take the CUs before the shrink's many small ones fill
    // them.  (Under graph capture the side stream joins the capture through
    // the fork event.)
    hipStream_t ss = s;
    if (mid) {
        BDL_HIP(hipEventRecord(P->fork_ev, s));
        if (ev) BDL_HIP(hipEventRecord(ev[4], s));
        BDL_HIP(bdl::launch_gemm_mid(fa, s));
        if (ev) BDL_HIP(hipEventRecord(ev[5], s));
        BDL_HIP(hipStreamWaitEvent(P->side_stream, P->fork_ev, 0));
        ss = P->side_stream;
    }
    if (ev) BDL_HIP(hipEventRecord(ev[2], ss));
    BDL_HIP(bdl::launch_shrink(fa, k.smb, k.snb, ss));
    if (ev) BDL_HIP(hipEventRecord(ev[3], ss));
    if (mid) BDL_HIP(hipEventRecord(P->join_ev, ss));
    if (!mid) {
        // the fused expand of the 64-row and large tiles reads Z: after the shrink
        if (ev) BDL_HIP(hipEventRecord(ev[4], s));
        if (big)
            BDL_HIP(bdl::launch_gemm_big(fa, s));
        else
            BDL_HIP(bdl::launch_gemm(fa, k.gmb, k.gnb, s));
        if (ev) BDL_HIP(hipEventRecord(ev[5], s));
    }
    if (mid) BDL_HIP(hipStreamWaitEvent(s, P->join_ev, 0));
    if (ev) BDL_HIP(hipEventRecord(ev[6], s));
    if (mid) BDL_HIP(bdl::launch_mid_epi(fa, s));
    if (ev) BDL_HIP(hipEventRecord(ev[7], s));
    P->last_path = big ? BDLORA_PATH_LARGE : (mid ? BDLORA_PATH_MEDIUM : BDLORA_PATH_TILE64);
    return BDLORA_OK;
}

// The batch's adapters: device ids, or host segments checked here (tiling
// 0..T-1 in order, every slot loaded or -1) and copied into *B.
static int read_batch(bdlora_pool_t P, const int32_t* ids, const bdlora_segments* sg, int T, Batch* B) {
    if ((ids != nullptr) == (sg != nullptr)) return fail(BDLORA_ERR_INVALID_ARG, "give exactly one of ids and segs");
    if (ids) {
        B->ids = ids;
        return BDLORA_OK;
    }
    const int n = sg->n_seg;
    if (n < 1 || n > bdl::kMaxSeg) return fail(BDLORA_ERR_INVALID_ARG, "n_seg must be 1..BDLORA_MAX_SEGMENTS");
    if (!sg->start || !sg->len || !sg->slot) return fail(BDLORA_ERR_INVALID_ARG, "null segment array");
    long long next = 0;
    bool bad = false;
    for (int i = 0; i < n; ++i) {
        if (sg->start[i] != next || sg->len[i] < 1)
            return fail(BDLORA_ERR_INVALID_ARG, "segments must tile 0..T-1 in order (segment " + std::to_string(i) + ")");
        next += sg->len[i];
        const int a = sg->slot[i];
        if (a != -1 && (a < 0 || a >= P->L.max_slots || !P->h_loaded[a])) bad = true;
        B->seg_start[i] = sg->start[i];
        B->seg_slot[i] = a;
    }
    if (next != T) return fail(BDLORA_ERR_INVALID_ARG, "segment lengths do not add up to T");
    if (bad) return fail(BDLORA_ERR_BAD_ADAPTER, "a segment names no loaded adapter slot");
    B->ids = nullptr;
    B->n_seg = n;
    return BDLORA_OK;
}

// Argument checks shared by the layer entry points.
static int check_layer_args(bdlora_pool_t P, int n, const int32_t* projs, const void* const* X,
                            const void* const* W, void* const* out, int T) {
    if (!P) return fail(BDLORA_ERR_INVALID_ARG, "null pool");
    const Layout& L = P->L;
    if (n < 1 || n > BDLORA_MAX_PROJS) return fail(BDLORA_ERR_INVALID_ARG, "n must be 1..8");
    if (!projs || !X || !W || !out) return fail(BDLORA_ERR_INVALID_ARG, "null pointer array");
    if (T < 0 || T > L.max_tokens) return fail(BDLORA_ERR_SHAPE, "T outside 0..max_tokens");
    bool seen[bdl::kMaxProjs] = {};
    for (int i = 0; i < n; ++i) {
        if (projs[i] < 0 || projs[i] >= L.n_projs) return fail(BDLORA_ERR_INVALID_ARG, "projection index out of range");
        if (seen[projs[i]]) return fail(BDLORA_ERR_INVALID_ARG, "projection listed twice");
        seen[projs[i]] = true;
        if (T > 0 && (!X[i] || !W[i] || !out[i])) return fail(BDLORA_ERR_INVALID_ARG, "null tensor pointer");
        if (T > 0 && (!aligned16(X[i]) || !aligned16(W[i]) || !aligned16(out[i])))
            return fail(BDLORA_ERR_INVALID_ARG, "X, W and out must be 16-byte aligned");
    }
    return BDLORA_OK;
}

int bdlora_forward_layer(bdlora_pool_t P, int32_t n, const int32_t* projs, const void* const* X,
                         const void* const* W, void* const* out, const int32_t* ids, const bdlora_segments* segs,
                         int32_t T, void* stream) {
    if (int rc = check_layer_args(P, n, projs, X, W, out, T)) return rc;
    const Layout& L = P->L;
    if (T == 0) return BDLORA_OK;
    Batch B;
    if (int rc = read_batch(P, ids, segs, T, &B)) return rc;
    DeviceGuard guard(P->device);
    if (!guard.ok) return fail(BDLORA_ERR_HIP, "hipSetDevice failed");
    hipStream_t s = (hipStream_t)stream;

    if (use_decode(L, T)) return forward_decode(P, n, projs, X, W, out, B, T, s, pool_dec_ws(P, n, projs));
    return forward_prefill(P, n, projs, X, W, out, B, T, s);
}

int bdlora_forward_layer_static(bdlora_pool_t P, int32_t n, const int32_t* projs, const void* const* X,
                                const void* const* W, void* const* out, const int32_t* ids,
                                const bdlora_segments* segs, int32_t T, void* stream) {
    if (int rc = check_layer_args(P, n, projs, X, W, out, T)) return rc;
    if (T == 0) return BDLORA_OK;
    if (T > bdl::kDecodeMaxT)
        return fail(BDLORA_ERR_SHAPE, "the static-scratch forward takes decode batches (T <= BDLORA_DECODE_MAX_T)");
    Batch B;
    if (int rc = read_batch(P, ids, segs, T, &B)) return rc;
    char* base = static_cast<char*>(bdl::static_scratch(P->device));
    if (!base)
        return fail(BDLORA_ERR_HIP, std::string("static scratch address not available on this device: ") +
                                        hipGetErrorString(P->static_err));
    // the array carved in 256-byte aligned pieces: plan tables, packed
    // activations per projection of the call, then the partial tiles
    long long off = 0;
    auto take = [&](long long bytes) {
        char* p = base + off;
        off = round_up(off + bytes, 256);
        return p;
    };
    DecWs w;
    w.meta = reinterpret_cast<int*>(take(16));
    w.vid = reinterpret_cast<int*>(take(4LL * bdl::kDecodeMaxT));
    w.tr8 = reinterpret_cast<int*>(take(4LL * bdl::kDecodeMaxT));
    w.tgrp = reinterpret_cast<int*>(take(4LL * bdl::kDecodeMaxT));
    w.gslot = reinterpret_cast<int*>(take(4LL * (bdl::kDecodeMaxT + 1)));
    w.gr8 = reinterpret_cast<int*>(take(4LL * (bdl::kDecodeMaxT + 1)));
    for (int i = 0; i < n; ++i) w.Xp[i] = reinterpret_cast<uint16_t*>(take(round_up(T, 16) * P->L.proj[projs[i]].K * 2LL));
    if (off > bdl::kStaticScratchBytes)
        return fail(BDLORA_ERR_SHAPE, "the call's packed activations need " + std::to_string(off) +
                                          " bytes, more than BDLORA_STATIC_SCRATCH_BYTES");
    w.part = nullptr;
    w.arena = base + off;
    w.arena_bytes = bdl::kStaticScratchBytes - off;
    DeviceGuard guard(P->device);
    if (!guard.ok) return fail(BDLORA_ERR_HIP, "hipSetDevice failed");
    return forward_decode(P, n, projs, X, W, out, B, T, (hipStream_t)stream, w);
}

int bdlora_forward_shard(bdlora_pool_t P, int32_t proj, const void* X, const void* W, const int32_t* ids,
                         const bdlora_segments* segs, int32_t T, void* out, void* stream) {
    const void* xs[1] = {X};
    const void* ws[1] = {W};
    void* os[1] = {out};
    int32_t pr[1] = {proj};
    return bdlora_forward_layer(P, 1, pr, xs, ws, os, ids, segs, T, stream);
}

int bdlora_forward_mlp(bdlora_pool_t P, int32_t act, const int32_t* first, int32_t down, const void* X,
                       const void* const* W_first, const void* W_down, void* out, const int32_t* ids,
                       const bdlora_segments* segs, int32_t T, void* stream) {
    if (!P) return fail(BDLORA_ERR_INVALID_ARG, "null pool");
    const Layout& L = P->L;
    if (act != BDLORA_ACT_NONE && act != BDLORA_ACT_SILU_MUL) return fail(BDLORA_ERR_INVALID_ARG, "unknown act");
    const int nf = act == BDLORA_ACT_SILU_MUL ? 2 : 1;
    if (!first || !W_first) return fail(BDLORA_ERR_INVALID_ARG, "null pointer array");
    if (T < 0 || T > L.max_tokens) return fail(BDLORA_ERR_SHAPE, "T outside 0..max_tokens");
    if (down < 0 || down >= L.n_projs) return fail(BDLORA_ERR_INVALID_ARG, "projection index out of range");
    for (int j = 0; j < nf; ++j) {
        if (first[j] < 0 || first[j] >= L.n_projs) return fail(BDLORA_ERR_INVALID_ARG, "projection index out of range");
        if (first[j] == down || (j == 1 && first[1] == first[0]))
            return fail(BDLORA_ERR_INVALID_ARG, "projection listed twice");
        if (L.proj[first[j]].kind != BDLORA_COLUMN || L.proj[first[j]].S != 1)
            return fail(BDLORA_ERR_INVALID_ARG, "first projections must be single-slice column projections");
        if (L.proj[first[j]].N != L.proj[down].K || L.proj[first[j]].K != L.proj[first[0]].K)
            return fail(BDLORA_ERR_SHAPE, "first projections' width must equal down's d_in");
    }
    if (L.proj[down].kind != BDLORA_ROW) return fail(BDLORA_ERR_INVALID_ARG, "down must be a row projection");
    if (T == 0) return BDLORA_OK;
    if (!X || !W_down || !out) return fail(BDLORA_ERR_INVALID_ARG, "null tensor pointer");
    for (int j = 0; j < nf; ++j)
        if (!W_first[j] || !aligned16(W_first[j])) return fail(BDLORA_ERR_INVALID_ARG, "W must be 16-byte aligned");
    if (!aligned16(X) || !aligned16(W_down) || !aligned16(out))
        return fail(BDLORA_ERR_INVALID_ARG, "X, W and out must be 16-byte aligned");
    Batch B;
    if (int rc = read_batch(P, ids, segs, T, &B)) return rc;
    DeviceGuard guard(P->device);
    if (!guard.ok) return fail(BDLORA_ERR_HIP, "hipSetDevice failed");
    hipStream_t s = (hipStream_t)stream;
    const int Ni = L.proj[down].K;                 // intermediate width d_I / N
    uint16_t* h = P->d_Xp[down];                   // H, packed as down's input
    const void* xs[2] = {X, X};
    const int32_t dn[1] = {down};
    const void* wd[1] = {W_down};
    void* od[1] = {out};
    if (use_decode(L, T)) {
        // first projections: their epilogue writes H packed; down reuses the plan
        DecMode m1;
        m1.mlp_act = act;
        m1.h_dst = h;
        m1.h_KS = Ni / 32;
        void* none[2] = {nullptr, nullptr};
        int rc = forward_decode(P, nf, first, xs, W_first, none, B, T, s, pool_dec_ws(P, nf, first), m1);
        if (rc) return rc;
        DecMode m2;
        m2.prep = false;
        return forward_decode(P, 1, dn, xs, wd, od, B, T, s, pool_dec_ws(P, 1, dn), m2);
    }
    // larger batches: the first projections' epilogue writes H (bf16,
    // packed as down's input) on the large-tile and medium-batch paths; on
    // the 64-row path they write fp32 to the pool's workspace and a pack
    // launch forms H.  Then down reads H in place.
    MlpOut mo;
    mo.act = act;
    mo.h = h;
    mo.h_KS = Ni / 32;
    mo.f32[0] = P->d_mlp;
    mo.f32[1] = P->d_mlp + (size_t)T * Ni;
    void* none[2] = {nullptr, nullptr};
    int rc = forward_prefill(P, nf, first, xs, W_first, none, B, T, s, true, &mo);
    if (rc) return rc;
    if (P->last_path == BDLORA_PATH_TILE64)
        BDL_HIP(bdl::launch_mlp_pack(mo.f32[0], act == BDLORA_ACT_SILU_MUL ? mo.f32[1] : nullptr, h, T, Ni, s));
    return forward_prefill(P, 1, dn, xs, wd, od, B, T, s, false);
}

int bdlora_plan_device(bdlora_pool_t P, const int32_t* ids, int32_t T, int32_t* vid, int32_t* gslot, int32_t* gstart,
                       int32_t* gcount, int32_t* perm, int32_t* n_groups, void* stream) {
    if (!P) return fail(BDLORA_ERR_INVALID_ARG, "null pool");
    if (T < 0 || T > P->L.max_tokens) return fail(BDLORA_ERR_SHAPE, "T outside 0..max_tokens");
    if (!n_groups || (T > 0 && (!ids || !vid || !gslot || !gstart || !gcount || !perm)))
        return fail(BDLORA_ERR_INVALID_ARG, "null pointer");
    DeviceGuard guard(P->device);
    if (!guard.ok) return fail(BDLORA_ERR_HIP, "hipSetDevice failed");
    hipStream_t s = (hipStream_t)stream;
    bdl::PrepArgs pa;
    Batch B;
    B.ids = ids;
    fill_plan_args(P, B, T, &pa, pick_shapes(T));
    BDL_HIP(bdl::launch_prep(pa, s));
    const int G = std::min(T, P->L.max_slots);
    if (T > 0) {
        BDL_HIP(hipMemcpyAsync(vid, P->d_vid, (size_t)T * 4, hipMemcpyDeviceToDevice, s));
        BDL_HIP(hipMemcpyAsync(perm, P->d_perm, (size_t)T * 4, hipMemcpyDeviceToDevice, s));
    }
    if (G > 0) {
        BDL_HIP(hipMemcpyAsync(gslot, P->d_gslot, (size_t)G * 4, hipMemcpyDeviceToDevice, s));
        BDL_HIP(hipMemcpyAsync(gstart, P->d_gstart, (size_t)G * 4, hipMemcpyDeviceToDevice, s));
        BDL_HIP(hipMemcpyAsync(gcount, P->d_gcount, (size_t)G * 4, hipMemcpyDeviceToDevice, s));
    }
    BDL_HIP(hipMemcpyAsync(n_groups, P->d_meta, 4, hipMemcpyDeviceToDevice, s));
    return BDLORA_OK;
}

int bdlora_pack_weight(const void* W, void* W_packed, int32_t N, int32_t K, void* stream) {
    if (!W || !W_packed) return fail(BDLORA_ERR_INVALID_ARG, "null pointer");
    if (W == W_packed) return fail(BDLORA_ERR_INVALID_ARG, "packing cannot run in place");
    if (N < 16 || N % 16 || K < 32 || K % 32) return fail(BDLORA_ERR_SHAPE, "N must be a multiple of 16, K of 32");
    if (!aligned16(W) || !aligned16(W_packed)) return fail(BDLORA_ERR_INVALID_ARG, "pointers must be 16-byte aligned");
    BDL_HIP(bdl::launch_pack_rows((const uint16_t*)W, (uint16_t*)W_packed, N, K, (hipStream_t)stream));
    return BDLORA_OK;
}

size_t bdlora_packed_weight_bytes(int32_t weight_format, int32_t N, int32_t K) {
    if (N < 16 || K < 32 || N > (1 << 20) || K > (1 << 20)) return 0;
    if (weight_format == BDLORA_WEIGHT_BF16)
        return N % 16 || K % 32 ? 0 : (size_t)N * K * 2;
    if (weight_format == BDLORA_WEIGHT_INT4_G128)
        return N % 64 || K % 128 ? 0 : (size_t)N * K / 2 + (size_t)N * (K / 128) * 2;
    return 0;
}

int bdlora_pack_weight_int4(const void* q, const void* scales, void* W_packed, int32_t N, int32_t K,
                            void* stream) {
    if (!q || !scales || !W_packed) return fail(BDLORA_ERR_INVALID_ARG, "null pointer");
    if (N < 64 || N % 64 || K < 128 || K % 128 || N > (1 << 20) || K > (1 << 20))
        return fail(BDLORA_ERR_SHAPE, "N must be a multiple of 64, K of 128");
    if (!aligned16(W_packed)) return fail(BDLORA_ERR_INVALID_ARG, "W_packed must be 16-byte aligned");
    if (reinterpret_cast<uintptr_t>(scales) % 2) return fail(BDLORA_ERR_INVALID_ARG, "scales must be 2-byte aligned");
    const size_t bytes = bdlora_packed_weight_bytes(BDLORA_WEIGHT_INT4_G128, N, K);
    const char* d0 = static_cast<const char*>(W_packed);
    auto overlaps = [&](const void* p, size_t n) {
        const char* c = static_cast<const char*>(p);
        return c < d0 + bytes && d0 < c + n;
    };
    if (overlaps(q, (size_t)N * K / 2) || overlaps(scales, (size_t)N * (K / 128) * 2))
        return fail(BDLORA_ERR_INVALID_ARG, "packing cannot overlap its inputs");
    uint32_t* dw = static_cast<uint32_t*>(W_packed);
    uint16_t* ds = reinterpret_cast<uint16_t*>(static_cast<char*>(W_packed) + (size_t)N * K / 2);
    BDL_HIP(bdl::launch_pack_int4(static_cast<const uint8_t*>(q), static_cast<const uint16_t*>(scales), dw, ds, N, K,
                                  (hipStream_t)stream));
    return BDLORA_OK;
}

int bdlora_get_device_error(bdlora_pool_t P, void* stream, int32_t* flag) {
    if (!P || !flag) return fail(BDLORA_ERR_INVALID_ARG, "null argument");
    DeviceGuard guard(P->device);
    if (!guard.ok) return fail(BDLORA_ERR_HIP, "hipSetDevice failed");
    hipStream_t s = (hipStream_t)stream;
    int32_t v = 0;
    BDL_HIP(hipMemcpyAsync(&v, P->d_err, 4, hipMemcpyDeviceToHost, s));
    BDL_HIP(hipStreamSynchronize(s));
    const int32_t zero = 0;
    BDL_HIP(hipMemcpyAsync(P->d_err, &zero, 4, hipMemcpyHostToDevice, s));
    BDL_HIP(hipStreamSynchronize(s));
    *flag = v;
    return BDLORA_OK;
}

int bdlora_profile_begin(bdlora_pool_t P, int32_t n) {
    if (!P || n < 0 || n > 100000) return fail(BDLORA_ERR_INVALID_ARG, "bad arguments");
    DeviceGuard guard(P->device);
    if (!guard.ok) return fail(BDLORA_ERR_HIP, "hipSetDevice failed");
    while (P->prof_ev.size() < (size_t)n * kProfEvents) {
        hipEvent_t e;
        BDL_HIP(hipEventCreate(&e));
        P->prof_ev.push_back(e);
    }
    P->prof_left = n;
    P->prof_used = 0;
    return BDLORA_OK;
}

int bdlora_profile_end(bdlora_pool_t P, float* ms, int32_t* n) {
    if (!P || !ms || !n) return fail(BDLORA_ERR_INVALID_ARG, "null argument");
    DeviceGuard guard(P->device);
    if (!guard.ok) return fail(BDLORA_ERR_HIP, "hipSetDevice failed");
    double sum[kProfEvents / 2] = {};
    for (int i = 0; i < P->prof_used; ++i) {
        hipEvent_t* ev = &P->prof_ev[(size_t)i * kProfEvents];
        BDL_HIP(hipEventSynchronize(ev[kProfEvents - 1]));
        for (int k = 0; k < kProfEvents / 2; ++k) {
            float t = 0.f;
            BDL_HIP(hipEventElapsedTime(&t, ev[2 * k], ev[2 * k + 1]));
            sum[k] += t;
        }
    }
    for (int k = 0; k < kProfEvents / 2; ++k) ms[k] = P->prof_used ? (float)(sum[k] / P->prof_used) : 0.f;
    *n = P->prof_used;
    P->prof_left = 0;
    P->prof_used = 0;
    return BDLORA_OK;
}

int bdlora_last_path(bdlora_pool_t P, int32_t* path) {
    if (!P || !path) return fail(BDLORA_ERR_INVALID_ARG, "null argument");
    *path = P->last_path;
    return BDLORA_OK;
}

}  // extern "C"
