// Launch descriptors shared by the host side of the library and its kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bdl {

constexpr int kMaxProjs = 8;
constexpr int kMaxSlices = 4;
constexpr int kMaxSlots = 8192;
constexpr int kMaxRank8 = 128;      // largest supported rank, rounded up to 8

// One projection of a forward launch.
struct ProjLaunch {
    const uint16_t* X;        // [T x K]   bf16
    const uint16_t* W;        // [N x K]   bf16 (nn.Linear layout)
    uint16_t* out;            // [T x N]   bf16
    uint16_t* Z;              // [2 x max_tokens x zs] workspace: scale * X A per slice as a
                              // bf16 pair (hi plane, then lo plane at Z + zplane)
    long long zplane;         // elements between the hi and the lo plane
    int K, N, n_slices, zs;
    int slice_col[kMaxSlices + 1];   // first column of each slice; [n_slices] = N
    long long a_off, b_off;   // element offsets of A^T_cat and B^T_cat in a slot
    int tiles_n;              // base GEMM: column tiles of this projection
    int tile_base;            // base GEMM: first flattened tile of this projection
};

// Everything one forward launch needs (passed by value as a kernel argument).
struct FwdArgs {
    ProjLaunch p[kMaxProjs];
    int n_proj;
    int T;
    const uint16_t* pool;     // adapter slabs
    long long slot_stride;    // elements per slot
    int max_slots;
    int r8max;                // per-slice Z stride (elements)
    const int* r8;            // [max_slots] rank rounded up to 8 (0: none)
    const float* scale;       // [max_slots]
    const int* vid;           // [T] validated ids
    const int* perm;          // [T] tokens grouped by adapter
    const int* gslot;         // [groups]
    const int* gstart;        // [groups] start in perm
    const int* gcount;        // [groups]
    const int* gitem;         // [groups + 1] first shrink item of each group
    const int* meta;          // [0] groups, [1] shrink items
    int items_bound;          // shrink: upper bound on items per projection
    int cchunks;              // shrink: column chunks per item (upper bound)
    int mts;                  // shrink: rows per item
    int tiles_m;              // base GEMM: row tiles
    int total_tiles;          // base GEMM: flattened tiles over all projections
};

// Plan launch (one workgroup).
struct PlanArgs {
    const int* ids;
    int T;
    const int* loaded;
    int max_slots;
    int mts;
    int* vid;
    int* perm;
    int* gslot;
    int* gstart;
    int* gcount;
    int* gitem;
    int* meta;
    int* err;
};

// Host-side launchers (bdl_kernels.hip).
hipError_t launch_plan(const PlanArgs& a, hipStream_t s);
hipError_t launch_shrink(const FwdArgs& a, int mb, hipStream_t s);
hipError_t launch_gemm(const FwdArgs& a, int mb, int nb, hipStream_t s);
hipError_t launch_pack(uint16_t* dst_a, uint16_t* dst_b, const uint16_t* stage, int K, int n_slices,
                       const int* slice_out, int rank, int r8, hipStream_t s);
int gemm_tile_rows(int mb);
int gemm_tile_cols(int nb);
int shrink_tile_cols();

}  // namespace bdl
