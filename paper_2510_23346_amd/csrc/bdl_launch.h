// Launch descriptors shared by the host side of the library and its kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "bdlora.h"

namespace bdl {

constexpr int kMaxProjs = 8;
constexpr int kMaxSlices = 4;
constexpr int kMaxSlots = 8192;
constexpr int kMaxRank8 = 128;       // largest supported rank, rounded up to 8
constexpr int kPlanLdsTokens = 8192; // plan keeps validated ids in LDS up to this batch size
constexpr int kPlanWaveGroups = 256;  // plan: placement by all waves for at most this many adapters
constexpr int kPlanParMaxSlots = 4096; // ... in pools of at most this many slots (its LDS counts)
constexpr int kMaxSeg = BDLORA_MAX_SEGMENTS;   // segments of a batch given in run-length form
constexpr int kBigM = 256, kBigN = 256;   // output tile of the large-tile base GEMM (prefill)
constexpr int kBigPartSlots = 256;        // fp32 partial tiles of the large-tile GEMM's split tiles
constexpr int kBigPartElems = kBigM * kBigN;
constexpr int kMidMaxT = 256;             // medium-batch base GEMM: largest batch (all rows in one tile)
constexpr int kShrinkKP = 4;              // shrink k-ranges per item when split (range k on XCDs k, k + 4)
constexpr long long kShrinkPartElems = 8LL << 20;   // fp32 partials of the split shrink (32 MiB)

// One projection of a forward launch.
struct ProjLaunch {
    const uint16_t* X;        // [T x K] bf16 activations (row-major)
    const uint16_t* Xp;       // packed activations, fragment layout, rows padded to 16
    int x_rowmajor;           // large-tile and medium-batch paths: the shrink and the GEMM read X
                              // (row-major, rows gathered by token) and Xp is not written; else Xp
    const uint16_t* W;        // packed base weight, fragment layout ([N x K] nn.Linear rows)
    const uint16_t* Ws;       // INT4 base: its scales (null for a bf16 base)
    uint16_t* out;            // [T x N] bf16
    float* out_f32;           // when set: the output in fp32 [T x N] instead of out
    uint16_t* Z;              // [2 x max_tokens x zs] workspace: scale * X A per slice as a
                              // bf16 pair (hi plane, then lo plane at Z + zplane)
    long long zplane;         // elements between the hi and the lo plane
    int K, N, n_slices, zs;
    int slice_col[kMaxSlices + 1];   // first column of each slice; [n_slices] = N
    long long a_off, b_off;   // element offsets of packed A^T_cat and of B^T_cat in a slot
    int tiles_n;              // base GEMM: column tiles of this projection
    int tile_base;            // base GEMM: first flattened tile (large tiles: work item) of this projection
    int ksplit;               // large-tile / medium-batch GEMM: k-ranges per tile (1: not split)
    int fix_base;             // large-tile GEMM: first split tile of this projection in the fix-up order
    int fix_count;            // large-tile GEMM: split tiles of this projection (0 when ksplit is 1)
    int part_base;            // large-tile GEMM: first partial tile of this projection's split tiles;
                              // medium-batch GEMM: first work item (= partial tile) of this projection
    int col_base;             // medium-batch GEMM: first 64-column epilogue tile of this projection
};

// Everything one forward launch needs (passed by value as a kernel argument).
struct FwdArgs {
    ProjLaunch p[kMaxProjs];
    int n_proj;
    int T;
    const uint16_t* pool;     // adapter slabs
    long long slot_stride;    // elements per slot
    int r8max;                // per-slice Z stride (elements)
    const float* scale;       // [max_slots]
    const int* vid;           // [T] validated ids
    const int* perm;          // [T] tokens grouped by adapter
    const int* rowtok;        // large-tile GEMM: token of each tile row (adapter order), or null
    const int* rowslot;       // medium-batch GEMM: (rank8 << 16) | slot of each such row, -1 for none
    const int4* items;        // shrink items {slot, first perm index, rows, r8}
    const int* meta;          // [1] number of shrink items
    int items_bound;          // shrink: upper bound on items
    int cchunks;              // shrink: column chunks per item (upper bound)
    int shrink_kp;            // shrink: k-ranges per item (1, or kShrinkKP: fp32 partials in
                              // shrinkpart that a second launch sums into Z)
    int* queue;               // unsplit shrink: unit counter, zeroed by the plan (meta[2])
    int sorder[kMaxProjs];    // unsplit shrink: projections in unit order (longest K first)
    float* shrinkpart;        // split shrink: fp32 partials (kShrinkPartElems)
    const int* tile_oct;      // expand octet codes per row tile (-1 padded)
    int oct_cap;              // entries per row tile in tile_oct
    int tiles_m;              // base GEMM: row tiles
    int total_tiles;          // base GEMM: flattened tiles (large tiles: work items) over all projections
    float* bigpart;           // large-tile GEMM: fp32 partials of split tiles (kBigPartSlots tiles)
    int fixup;                // large-tile GEMM: 0 main launch, 1 fix-up launch of the split tiles
    int total_fix;            // large-tile GEMM: split tiles over all projections
    int mid_rb, mid_nb;       // medium-batch GEMM: 16-row blocks per tile, 16-column blocks per wave
    int mid_items;            // medium-batch GEMM: work items (tile x k-range) over all projections
    int mid_col_tiles;        // medium-batch GEMM: 64-column epilogue tiles over all projections
    int max_slots;            // pool slots
    // MLP intermediate (large-tile and medium-batch launches of the MLP's
    // first projections): -1 writes out / out_f32; BDLORA_ACT_NONE writes
    // H = projection 0's output, BDLORA_ACT_SILU_MUL H = silu(projection 0)
    // * projection 1 (gate and up of equal shape; their tiles are paired so
    // one workgroup holds both), in bf16 into h_dst in the fragment layout of
    // the second projection's input (rows = tokens, h_KS k-steps)
    int mlp_act;
    uint16_t* h_dst;
    int h_KS;
};

// Activation packing job of the prep launch.
struct PackJob {
    const uint16_t* src;      // [rows x K] row-major
    uint16_t* dst;            // fragment layout, rows padded to a multiple of 16
    int rows, K;
    int frag_base;            // first fragment of this job in the launch's numbering
};

// Prep launch: workgroup 0 plans the batch, the others pack activations.
struct PrepArgs {
    const int* ids;           // [T] per-token ids, or null: the batch is given by the segments below
    int T;
    int n_seg;                // segments (ids null): token t takes seg_slot[i] of the last i with
    int seg_start[kMaxSeg];   // seg_start[i] <= t (the host checked that they tile 0..T-1)
    int seg_slot[kMaxSeg];
    int act_max;              // decode plan: adapters past this many (slot order) are treated as
                              // none and raise *err (the decode launches' bound); -1: no bound
    const int* loaded;
    const int* r8;            // [max_slots]
    int max_slots;
    int mts;                  // shrink rows per item
    int gemm_mt;              // base GEMM row tile (<= 64)
    int oct_cap;
    int* vid;
    int* tr8;                 // [T] rank (padded to 8) of each token's adapter, 0 if none
    int* tgrp;                // [T] group index of each token's adapter, -1 if none (optional)
    int* perm;
    int* rowtok;              // optional [T]: the adapted tokens in perm order, then the others in order
    int* rowslot;             // optional [T], with rowtok: (rank8 << 16) | slot of each row's adapter, -1 for none
    int oct_perm;             // 1: octet lists for the 64-row blocks of rowtok order (large-tile GEMM)
    int* gslot;
    int* gr8;                 // decode plan (optional): padded rank of each adapter in use
    int* gstart;
    int* gcount;
    int4* items;
    int* tile_oct;
    int* meta;                // [0] groups, [1] shrink items, [2] the shrink's unit counter (zeroed)
    int* err;
    PackJob jobs[kMaxProjs];
    int n_jobs;
    int total_frags;
    int decode_plan;          // T <= 64: one wave writes vid, tr8, tgrp, gslot, meta only
};

// ---- decode path (T <= kDecodeMaxT) ----------------------------------------
// The main launch is one split-K GEMM of the packed activations against a
// virtual column list per projection: the W_s column blocks (16 columns
// each), then for every adapter the batch uses (in group order) the blocks of
// its A^T_cat.  Work is counted in units of one 16-column block times one
// 32-wide k-step; groups of 4 consecutive blocks are cut into k-ranges so
// that every workgroup of the launch gets the same number of units.
constexpr int kDecodeMaxT = BDLORA_DECODE_MAX_T;
constexpr int kDecMaxGrid = 1024;    // most workgroups of the main launch
constexpr int kPartElems = 64 * 64;  // fp32 partial tile: 64 rows x 64 virtual columns

struct DecProj {
    const uint16_t* X;        // the caller's activations [T x K], row-major (batches of at most 16
                              // tokens planned in the main launch); else null and Xp is read
    const uint16_t* Xp;       // packed activations (fragment layout)
    const uint16_t* W;        // packed base weight
    const uint16_t* Ws;       // INT4 base: its scales (null for a bf16 base)
    uint16_t* out;            // [T x N] bf16
    int K, N, n_slices;
    int slice_col[kMaxSlices + 1];
    long long a_off, b_off;
    int nWb;                  // W column blocks (N / 16)
    int nbA;                  // A^T_cat blocks per adapter (rows padded to 16)
    int tile_base;            // first epilogue tile (64 output columns) of this projection
};

struct DecArgs {
    // Schedule of the main launch, computed by the host for act_max adapter
    // positions: projection p's units start at sub[p] (sub[n_proj] = all
    // units) and its groups at sgb[p]; it has snb[p] virtual blocks and
    // sks[p] k-steps.  Kept first and compact so that a workgroup reads it
    // with a few scalar loads.
    unsigned units;
    unsigned sub[kMaxProjs];
    int sgb[kMaxProjs], snb[kMaxProjs], sks[kMaxProjs];
    int stb[kMaxProjs];       // first epilogue tile of each projection
    DecProj p[kMaxProjs];
    int n_proj;
    int T;
    const uint16_t* pool;
    long long slot_stride;
    const float* scale;       // [max_slots]
    // The batch's plan.  plan = 0: the prep launch wrote it into the tables
    // below.  plan = 1 (batches of at most 16 tokens): every wave of the main
    // launch computes it from the batch (ids, or segments) and the slot
    // tables, and the first wave of workgroup 0 stores the tables below.
    int plan;
    const int* ids;           // [T] per-token slot ids, or null: the segments below
    int n_seg;                // segments (ids null): token t takes seg_slot[i] of the last i with
    int seg_start[kDecodeMaxT];   // seg_start[i] <= t (the host checked that they tile 0..T-1)
    int seg_slot[kDecodeMaxT];
    const int* loaded;        // [max_slots] nonzero: the slot holds an adapter
    const int* r8;            // [max_slots] padded rank of each slot
    int max_slots;
    int* vid;                 // [T] validated ids
    int* tr8;                 // [T] padded rank of each token's adapter (0: none)
    int* tgrp;                // [T] group (adapter in use) index of each token, -1: none
    int* gslot;               // [groups] slot of each adapter in use
    int* gr8;                 // [groups] its rank padded to 8 (its A^T blocks: n_slices gr8 / 16,
                              // rounded up; positions past them hold no data)
    int* meta;                // [0] number of adapters in use (n_act)
    int act_max;              // adapter positions in the column lists: the host's bound on n_act;
                              // the plan treats adapters past it (slot order) as none and raises *err
    float* part;              // partial tiles: slot g + b for group g and workgroup b
    int part_slots;
    int main_grid;            // workgroups of the main launch
    int tiles;                // epilogue tiles over all projections
    int* err;                 // sticky error flag
    int mlp_act;              // -1: write out; else write the MLP intermediate H (BDLORA_ACT_*)
    uint16_t* h_dst;          // H in the fragment layout of the second projection's input
    int h_KS;                 // k-steps of that layout (second projection's d_in / 32)
};

// Host-side launchers (bdl_kernels.hip, bdl_prep.hip, bdl_decode.hip).
hipError_t launch_dec_main(const DecArgs& a, int mb, hipStream_t s);
hipError_t launch_dec_epi(const DecArgs& a, hipStream_t s);
hipError_t launch_prep(const PrepArgs& a, hipStream_t s);
hipError_t launch_shrink(const FwdArgs& a, int mb, int nb, hipStream_t s);
hipError_t launch_gemm(const FwdArgs& a, int mb, int nb, hipStream_t s);
hipError_t launch_gemm_big(const FwdArgs& a, hipStream_t s);
hipError_t launch_gemm_mid(const FwdArgs& a, hipStream_t s);
hipError_t launch_mid_epi(const FwdArgs& a, hipStream_t s);
hipError_t launch_pack_adapter(uint16_t* dst_a, uint16_t* dst_b, const uint16_t* stage, int K,
                               int n_slices, const int* slice_out, int rank, int r8, hipStream_t s);
hipError_t launch_pack_rows(const uint16_t* src, uint16_t* dst, int rows, int K, hipStream_t s);
// rank and scale tables of up to kMaxSlotBatch consecutive slots (kernel argument)
constexpr int kMaxSlotBatch = 64;
struct SlotBatch {
    int first, n;
    int r8[kMaxSlotBatch];
    float scale[kMaxSlotBatch];
};
hipError_t launch_set_slots(int* r8, float* scale, int* loaded, const SlotBatch& b, hipStream_t s);
hipError_t launch_pack_int4(const uint8_t* q, const uint16_t* scales, uint32_t* dst_w, uint16_t* dst_s, int N,
                            int K, hipStream_t s);
hipError_t launch_mlp_pack(const float* G, const float* U, uint16_t* dst, int T, int N, hipStream_t s);

// Static scratch of the allocation-free decode entry point (bdl_static.hip).
constexpr long long kStaticScratchBytes = BDLORA_STATIC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;
// Take the address of the current device's copy (call once per device, with
// it current; later calls return at once).
hipError_t static_scratch_init(int device);
// That address (null before static_scratch_init succeeded on the device).
void* static_scratch(int device);

}  // namespace bdl
