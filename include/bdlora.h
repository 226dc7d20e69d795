/*
 * bdlora.h -- C ABI of the MI355X (gfx950) block-diagonal LoRA shard library.
 *
 * What it computes.  One GPU's tensor-parallel share of a LoRA-augmented
 * projection, for a batch in which every token names its own adapter
 * (unmerged multi-adapter serving, paper Sec. 1; the BD-LoRA sharding of
 * Sec. 3 and Fig. 3; the per-device steps of Alg. 1 and Alg. 2):
 *
 *     out[t, :] = X[t, :] W_s^T + scale_a * (X[t, :] A_{s,a}) B_{s,a},  a = id(t)
 *
 * Column-parallel projections (q/k/v, gate, up): X is the replicated input,
 * A_{s,a} is the shard's column slice of A and B_{s,a} the shard's diagonal
 * block of the block-diagonal B, so the LoRA term lands on the shard's own
 * output columns.  Row-parallel projections (o, down): X is the shard's input
 * slice, A_{s,a} the shard's diagonal block of the block-diagonal A and
 * B_{s,a} the shard's row slice of B; `out` is then a partial sum that the
 * base model's all-reduce would add up (not run by this library).  A
 * projection may have up to 4 slices (q, k, v): each slice has its own
 * adapter factors and its outputs sit side by side.
 *
 * Conventions.
 *  - Element type of X, W_s, out and of adapter factors: bfloat16, passed as
 *    16-bit patterns (uint16_t on the host, any 2-byte type on the device).
 *    Products accumulate in fp32; out is rounded once to bf16 (nearest-even).
 *  - Layouts.  X: [T x d_in] row-major.  out: [T x d_out_s] row-major,
 *    slices side by side.  Base weights are packed once, before serving, by
 *    bdlora_pack_weight from the nn.Linear layout [d_out_s x d_in] into the
 *    matrix-core fragment layout the kernels stream (same size); forward
 *    calls take the packed weight.  Adapter factors are given in the paper's
 *    layout: A: [d_in x rank], B: [rank x slice_out] per slice.
 *  - Adapter ids: int32, one per token; -1 = no adapter (base only).  An id
 *    that is out of range or names an empty slot is treated as -1 and raises
 *    the pool's sticky device error flag (see bdlora_get_device_error).
 *  - Device pointers are caller-owned and must stay valid until the work
 *    enqueued on `stream` has finished.  `stream` is a hipStream_t (NULL =
 *    the default stream).  Forward calls only enqueue; they never block.
 *  - A pool owns the adapter memory and a workspace sized at creation.  All
 *    forward calls on one pool must be issued on one stream (the workspace is
 *    shared); use one pool per stream otherwise.  Loading or unloading an
 *    adapter must not overlap a forward that uses it.
 *  - Every int-returning call returns a status code below; on failure
 *    bdlora_last_error() gives a message (thread-local).
 */
#ifndef BDLORA_H
#define BDLORA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define BDLORA_OK               0
#define BDLORA_ERR_INVALID_ARG (-1)  /* null pointer, bad slot, bad value      */
#define BDLORA_ERR_OOM         (-2)  /* device or host allocation failed       */
#define BDLORA_ERR_BAD_ADAPTER (-3)  /* host-side id names no loaded adapter   */
#define BDLORA_ERR_SHAPE       (-4)  /* sizes the kernels do not support       */
#define BDLORA_ERR_HIP         (-5)  /* a HIP runtime call failed              */
#define BDLORA_ERR_UNSUPPORTED (-6)  /* no gfx950 device / feature missing     */

#define BDLORA_COLUMN 0
#define BDLORA_ROW    1
#define BDLORA_MAX_SLICES 4
#define BDLORA_MAX_PROJS  8
#define BDLORA_MAX_SLOTS  8192
#define BDLORA_MAX_RANK   128
/* Batches of at most this many tokens take the decode launch sequence (plan
 * and packing, K-split shrink and base partials, epilogue); larger ones take
 * the prefill sequence (plan and packing, shrink, base product with the
 * expand fused in, or for medium batches on large layers base partials and
 * an epilogue; see bdlora_last_path). */
#define BDLORA_DECODE_MAX_T 64
/* Decode batches skip the plan and packing launch when T <= 16, or when
 * T <= BDLORA_DECODE_PLAN_IN_MAIN_T and T x (the sum of d_in over the
 * call's projections) x 2 bytes <= BDLORA_DECODE_PLAN_IN_MAIN_BYTES: every
 * wave of the K-split launch then plans the batch from the ids (or
 * segments) itself and gathers the caller's row-major activations, which
 * slows that launch more the more activation bytes it gathers. */
#define BDLORA_DECODE_PLAN_IN_MAIN_T 32
#define BDLORA_DECODE_PLAN_IN_MAIN_BYTES 1572864
/* Largest number of segments a bdlora_segments batch may have (the segments
 * travel with the launch, by value). */
#define BDLORA_MAX_SEGMENTS 256
/* Activation between the two projections of bdlora_forward_mlp. */
#define BDLORA_ACT_NONE     0   /* H = first projection's output (Alg. 1)  */
#define BDLORA_ACT_SILU_MUL 1   /* H = silu(gate) * up (gated MLP)         */

/* Base weight formats (bdlora_proj_desc.weight_format).
 * BDLORA_WEIGHT_BF16: bf16 W_s, packed by bdlora_pack_weight.
 * BDLORA_WEIGHT_INT4_G128: weight-only INT4 base (the quantized backbone of
 *   Sec. 5.2 / App. F; activations and adapters stay bf16): symmetric INT4
 *   with one bf16 scale per output column and group of 128 inputs,
 *   W[n][k] = scale[n][k / 128] * q[n][k], q in -8..7, packed by
 *   bdlora_pack_weight_int4.  The kernels multiply the raw q by the bf16
 *   activations on the matrix cores and apply the scale in fp32 per k-step,
 *   so no dequantized weight is ever formed. */
#define BDLORA_WEIGHT_BF16      0
#define BDLORA_WEIGHT_INT4_G128 1

typedef struct bdlora_pool* bdlora_pool_t;

/* A batch given as segments instead of per-token ids (heterogeneous
 * batching, Sec. 2 on S-LoRA: the requests of a batch each name one
 * adapter, and a prefill request is a contiguous run of tokens).  Host
 * arrays of n_seg entries: segment i covers tokens start[i] ..
 * start[i] + len[i] - 1 and uses adapter slot[i] (-1 = no adapter).  The
 * segments must tile 0 .. T-1 in order: start[0] = 0, len[i] >= 1,
 * start[i+1] = start[i] + len[i], start[n_seg-1] + len[n_seg-1] = T.
 * 1 <= n_seg <= BDLORA_MAX_SEGMENTS.  Adjacent segments may name the same
 * slot.  The forward validates them on the host before anything is
 * enqueued and copies them into the launch, so the arrays may be freed or
 * reused as soon as the call returns (also under graph capture: a captured
 * forward replays the segments it was given). */
typedef struct {
    int32_t n_seg;
    const int32_t* start;
    const int32_t* len;
    const int32_t* slot;
} bdlora_segments;

/* One projection on one shard.  d_in: local input width (K), a multiple of
 * 32.  slice_out[i]: local output width of slice i, a multiple of 16.
 * kind only documents the sharding (BDLORA_COLUMN / BDLORA_ROW); both kinds
 * run the same per-shard computation (Alg. 1 first and second projection).
 * weight_format: BDLORA_WEIGHT_*; INT4 needs d_in a multiple of 128 and the
 * total output width a multiple of 64. */
typedef struct {
    int32_t kind;
    int32_t d_in;
    int32_t n_slices;
    int32_t slice_out[BDLORA_MAX_SLICES];
    int32_t weight_format;
} bdlora_proj_desc;

/* Create an adapter pool on HIP device `device` for the `n_projs`
 * projections described by `projs` (1..BDLORA_MAX_PROJS).  The pool has
 * adapter slots each sized for rank `max_rank` (0..BDLORA_MAX_RANK) on every
 * projection (bdlora_layout_slot_bytes bytes per slot), plus a workspace for
 * batches of up to `max_tokens` tokens.  Paper: the GPU-side adapter cache
 * of App. C.2 / App. F (adapters loaded once, reused by every batch).
 * Slot count and adapter memory:
 *   pool_bytes = 0:  max_slots slots (1..BDLORA_MAX_SLOTS);
 *   pool_bytes > 0, max_slots = 0: as many slots as pool_bytes holds
 *                    (at most BDLORA_MAX_SLOTS; OOM if not even one);
 *   pool_bytes > 0, max_slots > 0: max_slots slots, which must fit in
 *                    pool_bytes (else OOM, nothing allocated).
 * pool_bytes bounds the adapter slabs only; the workspace comes on top
 * (bdlora_pool_size reports both).  bdlora_pool_slots gives the count.
 * All memory is allocated here; forward calls allocate nothing.
 * On success *out receives the handle.  Errors: INVALID_ARG, SHAPE, OOM, HIP,
 * UNSUPPORTED (device is not gfx950). */
int bdlora_create_pool(const bdlora_proj_desc* projs, int32_t n_projs, int32_t max_slots,
                       int32_t max_rank, int32_t max_tokens, int64_t pool_bytes, int32_t device,
                       bdlora_pool_t* out);

/* Number of adapter slots of the pool.  Errors: INVALID_ARG. */
int bdlora_pool_slots(bdlora_pool_t pool, int32_t* slots);

/* Free every device and host resource of the pool (waits for its work). */
int bdlora_destroy_pool(bdlora_pool_t pool);

/* Copy one adapter into `slot` (0..max_slots-1) and pack it into the pool's
 * kernel layout on the device.  rank: 0..max_rank (0 = an adapter that adds
 * nothing).  scale: the factor of the LoRA term (rsLoRA-style gamma of Sec. 2;
 * BD-LoRA training uses alpha*sqrt(N)/sqrt(r), Sec. 3), finite.
 * A_host and B_host are arrays of host pointers indexed [proj][slice] in
 * projection-major order (slice index runs fastest): A is [d_in x rank] and
 * B is [rank x slice_out], bf16, row-major, the shard's own factors sliced as
 * in App. C.2 (column: A column block + B diagonal block; row: A diagonal
 * block + B row block).  Values must be finite.  The call is synchronous:
 * host buffers may be freed on return.  Replaces any adapter in the slot.
 * Errors: INVALID_ARG (bad slot/rank/scale, null pointer, non-finite value),
 * HIP. */
int bdlora_load_adapter(bdlora_pool_t pool, int32_t slot, int32_t rank, float scale,
                        const uint16_t* const* A_host, const uint16_t* const* B_host);

/* Adapter load pipeline (the per-request adapter loading of Sec. 5.2 / App. F:
 * an adapter that is not cached on the GPU is brought in before its request
 * runs; the time scales with its parameter count).  A host-side cache keeps
 * adapters already in the pool's slot layout; loading one is then a single
 * host-to-device copy of bdlora_slot_bytes(pool) bytes plus a table update,
 * both enqueued on the caller's stream so they can overlap forward calls that
 * use other slots on another stream. */

/* Bytes of one adapter slot of the pool (0 for a null pool). */
int64_t bdlora_slot_bytes(bdlora_pool_t pool);

/* Bytes of one adapter slot of any pool created with these projections and
 * max_rank (pure host function; App. C.2 compact storage, ranks padded to
 * multiples of 8).  Errors: INVALID_ARG, SHAPE. */
int bdlora_layout_slot_bytes(const bdlora_proj_desc* projs, int32_t n_projs, int32_t max_rank,
                             int64_t* bytes);

/* bdlora_pack_adapter_host without a pool (pure host code, no device
 * needed): packs one adapter for every pool created with these projections
 * and max_rank, into slab_host (bdlora_layout_slot_bytes bytes).  Lets a
 * process without a GPU prepare a host-side adapter cache.  Errors:
 * INVALID_ARG (bad rank, null pointer, non-finite value), SHAPE. */
int bdlora_pack_adapter_layout(const bdlora_proj_desc* projs, int32_t n_projs, int32_t max_rank,
                               int32_t rank, const uint16_t* const* A_host,
                               const uint16_t* const* B_host, void* slab_host);

/* Pack one adapter on the host into the pool's slot layout (for a host-side
 * cache): slab_host receives bdlora_slot_bytes(pool) bytes (padding zeroed).
 * rank, A_host and B_host as for bdlora_load_adapter.  Pure host code; the
 * result is byte-identical, in every region the kernels read, to what
 * bdlora_load_adapter writes on the device.  Errors: INVALID_ARG (bad rank,
 * null pointer, non-finite value). */
int bdlora_pack_adapter_host(bdlora_pool_t pool, int32_t rank, const uint16_t* const* A_host,
                             const uint16_t* const* B_host, void* slab_host);

/* Enqueue on `stream` the copy of a host-packed slab into `slot` and the
 * update of the slot's rank and scale; returns without waiting.  The whole
 * slot is copied (bdlora_slot_bytes: about 2 bytes per parameter for an
 * adapter of the pool's max_rank).  With
 * slab_host in pinned memory (hipHostMalloc, or a pinned torch tensor) the
 * copy is asynchronous; pageable memory is staged by the runtime.  The caller
 * keeps slab_host alive until the stream has passed the copy, orders forward
 * calls that use the slot after it (same stream, or an event), and must not
 * overwrite a slot that a forward in flight still reads.  Errors:
 * INVALID_ARG, HIP. */
int bdlora_load_adapter_packed(bdlora_pool_t pool, int32_t slot, int32_t rank, float scale,
                               const void* slab_host, void* stream);

/* As bdlora_load_adapter_packed for n (1..64) adapters into the consecutive
 * slots first_slot .. first_slot + n - 1: slabs_host holds their host-packed
 * slabs back to back (n * bdlora_slot_bytes bytes), ranks[i] and scales[i]
 * (host arrays) belong to slot first_slot + i.  One copy and one table
 * update for the whole batch.  Errors: INVALID_ARG, HIP. */
int bdlora_load_adapters_packed(bdlora_pool_t pool, int32_t first_slot, int32_t n, const int32_t* ranks,
                                const float* scales, const void* slabs_host, void* stream);

/* Mark `slot` empty; later ids naming it are invalid.  Errors: INVALID_ARG. */
int bdlora_unload_adapter(bdlora_pool_t pool, int32_t slot);

/* Pack a base weight W [N x K] (nn.Linear layout, row-major, bf16, device)
 * into W_packed (device, N*K elements, not overlapping W): 16-row blocks of
 * 32-wide k-steps, each stored as the 1 KB operand of one gfx950 bf16 MFMA
 * (element [(rb*(K/32) + ks)*512 + lane*8 + i] = W[16 rb + lane%16]
 * [32 ks + 8 (lane/16) + i]).  N: multiple of 16; K: multiple of 32.
 * Enqueued on `stream`.  Errors: INVALID_ARG, SHAPE, HIP. */
int bdlora_pack_weight(const void* W, void* W_packed, int32_t N, int32_t K, void* stream);

/* Bytes of a packed base weight [N x K] in format weight_format
 * (BDLORA_WEIGHT_*): 2 N K for bf16, N K / 2 + N K / 64 for INT4.
 * Returns 0 for an unknown format or sizes that format does not take. */
size_t bdlora_packed_weight_bytes(int32_t weight_format, int32_t N, int32_t K);

/* Pack an INT4 base weight (BDLORA_WEIGHT_INT4_G128) for forward calls.
 * q: device uint8 [N x K/2], row n of the nn.Linear layout, byte (n, j)
 * holding q[n][2j] + 8 in its low nibble and q[n][2j+1] + 8 in its high
 * nibble.  scales: device bf16 [N x K/128].  W_packed: device,
 * bdlora_packed_weight_bytes(BDLORA_WEIGHT_INT4_G128, N, K) bytes, 16-byte
 * aligned, not overlapping the inputs.  Layout: first N K / 2 bytes of
 * 32-bit words, word (rb (K/32) + ks) 64 + lane holding the 8 values
 * W[16 rb + lane%16][32 ks + 8 (lane/16) + i], value i in bits
 * 4 (i/2) + 16 (i%2) .. +3 (as q + 8); then the scales as bf16, entry
 * (rb (K/128) + g) 16 + c = scale[16 rb + c][g].  N: multiple of 64; K:
 * multiple of 128.  Enqueued on `stream`.  Errors: INVALID_ARG, SHAPE, HIP. */
int bdlora_pack_weight_int4(const void* q, const void* scales, void* W_packed, int32_t N, int32_t K,
                            void* stream);

/* One projection call (Alg. 2 on one device; Alg. 1 first or second
 * projection): out = X W_s^T + scale_a (X A_a) B_a per token.
 * proj: index into the pool's projection list.  X: device [T x d_in];
 * W: device, the base weight [d_out_s x d_in] packed by bdlora_pack_weight
 * (or bdlora_pack_weight_int4 for an INT4 projection); out: device
 * [T x d_out_s].  The batch's adapters come either as ids (device int32
 * [T], one per token; segs = NULL) or as segs (host segments, see
 * bdlora_segments; ids = NULL); exactly one of the two.  With segs an id
 * that names no loaded slot fails the call with BAD_ADAPTER before anything
 * is enqueued; with ids it is treated as -1 on the device and raises the
 * sticky device error flag.  Both forms give bit-identical outputs for the
 * same batch.  T: 0..max_tokens (T = 0 enqueues nothing).
 *
 * Graph capture.  A forward may be captured in a HIP graph; the replay
 * repeats the launches with the arguments of the capture.  The launch
 * geometry of a decode batch (T <= BDLORA_DECODE_MAX_T) given as ids covers
 * at most min(T, adapters loaded when the call is made) distinct adapters:
 * if a replay's ids use more distinct adapters than that (adapters loaded
 * after the capture), the tokens of the adapters past the bound (in
 * ascending slot order) get the base output only and the device error flag
 * is raised.  Recapture after loading adapters.  Larger batches have no such
 * bound, and segments, checked against the adapters loaded when the call is
 * made, stay within it.
 * Errors: INVALID_ARG, BAD_ADAPTER (segs only), SHAPE, HIP. */
int bdlora_forward_shard(bdlora_pool_t pool, int32_t proj, const void* X, const void* W,
                         const int32_t* ids, const bdlora_segments* segs, int32_t T, void* out,
                         void* stream);

/* Several projection calls that share the token batch and its ids or
 * segments (the projections of one decoder layer), enqueued as one plan,
 * one shrink and one base-plus-expand launch.  projs[i] indexes the pool's
 * projection list; X[i], W[i], out[i] are device pointers as for
 * bdlora_forward_shard (host arrays of n pointers).  n: 1..BDLORA_MAX_PROJS;
 * the same projection may not appear twice.  Errors: as
 * bdlora_forward_shard. */
int bdlora_forward_layer(bdlora_pool_t pool, int32_t n, const int32_t* projs,
                         const void* const* X, const void* const* W, void* const* out,
                         const int32_t* ids, const bdlora_segments* segs, int32_t T,
                         void* stream);

/* For callers that cannot allocate device memory during the call (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation):
 * bdlora_forward_layer for decode batches (1 <= T <= BDLORA_DECODE_MAX_T;
 * T = 0 enqueues nothing) whose per-batch scratch -- the plan's tables, the
 * packed activations and the fp32 partial tiles -- lives in a static device
 * array of BDLORA_STATIC_SCRATCH_BYTES that the library holds on every GPU it
 * runs on until the process ends, instead of in the pool's workspace.  The
 * call allocates nothing (no hipMalloc, no allocating library routine); the
 * pool still holds the adapters, their tables and the error flag.  Same
 * arguments, kernels, launch geometry and results (bit for bit) as
 * bdlora_forward_layer.  Every call on one GPU shares that GPU's array:
 * calls that overlap on one GPU (other streams, other pools, other threads)
 * race and must be serialized by the caller.  Nothing in the array has to
 * start at zero: every word a call reads was written earlier in that call.
 * Errors: as bdlora_forward_layer; SHAPE for T above BDLORA_DECODE_MAX_T or a
 * call whose scratch exceeds BDLORA_STATIC_SCRATCH_BYTES (the message gives
 * the sizes); HIP if the array's address could not be taken when the pool
 * was created. */
#define BDLORA_STATIC_SCRATCH_BYTES (32 << 20)
int bdlora_forward_layer_static(bdlora_pool_t pool, int32_t n, const int32_t* projs,
                                const void* const* X, const void* const* W, void* const* out,
                                const int32_t* ids, const bdlora_segments* segs, int32_t T,
                                void* stream);

/* One device's share of a BD-LoRA MLP (Alg. 1, App. B): the first
 * (column-parallel) projection(s), the intermediate H, then the
 * row-parallel projection `down`, whose output is the device's partial that
 * the base model's all-reduce would sum.  Alg. 1 chains the projections
 * directly (act = BDLORA_ACT_NONE: first[0] is one column projection and
 * H = its output); the gated MLP of the Llama models the paper serves
 * (Sec. 4) takes act = BDLORA_ACT_SILU_MUL with first[0] = gate and
 * first[1] = up, two column projections of equal width, and
 * H = silu(gate) * up.  Every projection adds its own BD-LoRA term per token
 * exactly as bdlora_forward_shard does.  H [T x d_in of down] is held in the
 * pool in bf16 (round to nearest even) and never leaves it; the first
 * projections' width must equal down's d_in.
 * X: device [T x d_in] bf16, shared by the first projections; W_first:
 * host array of 1 or 2 device pointers to packed weights; W_down: packed
 * weight of down; out: device [T x d_out of down]; ids (device int32 [T])
 * or segs (host segments), exactly one, as for bdlora_forward_shard.
 * T: 0..max_tokens.  Enqueued on `stream`; uses the pool's workspace, so
 * calls on one pool must share one stream.
 * Errors: INVALID_ARG (bad act, indices, kinds or null pointers),
 * BAD_ADAPTER (segs only), SHAPE (widths do not chain), HIP. */
int bdlora_forward_mlp(bdlora_pool_t pool, int32_t act, const int32_t* first, int32_t down,
                       const void* X, const void* const* W_first, const void* W_down, void* out,
                       const int32_t* ids, const bdlora_segments* segs, int32_t T, void* stream);

/* Host-side plan of a batch (the integer bookkeeping of heterogeneous
 * batching, Sec. 2 on S-LoRA), a pure host function: validates host ids
 * against `loaded` (max_slots flags, nonzero = slot holds an adapter) and
 * groups tokens by adapter.  Outputs (host arrays, caller-allocated):
 *   vid[T]          validated id per token (-1 for none),
 *   group_slot/group_start/group_count[n]  one entry per adapter in use,
 *                   slots ascending, starts into perm,
 *   perm[T]         tokens with an adapter, group after group, ascending
 *                   inside each group,
 *   *n_groups       number of groups.
 * group arrays must hold min(T, max_slots) entries.  Returns BAD_ADAPTER
 * (after filling the outputs, invalid ids mapped to -1) when some id other
 * than -1 names no loaded slot. */
int bdlora_build_plan(const int32_t* loaded, int32_t max_slots, const int32_t* ids_host, int32_t T,
                      int32_t* vid, int32_t* group_slot, int32_t* group_start,
                      int32_t* group_count, int32_t* perm, int32_t* n_groups);

/* Run the device plan step that every forward call runs first, and copy its
 * results to caller device buffers of the same shapes as bdlora_build_plan
 * (n_groups is a device int32).  Inside a group the device lists tokens in
 * ascending order as well.  Enqueued on `stream`.  Errors: INVALID_ARG,
 * SHAPE, HIP. */
int bdlora_plan_device(bdlora_pool_t pool, const int32_t* ids, int32_t T, int32_t* vid,
                       int32_t* group_slot, int32_t* group_start, int32_t* group_count,
                       int32_t* perm, int32_t* n_groups, void* stream);

/* Synchronise `stream`, return the sticky device error flag in *flag (1 if
 * some forward since the last call saw an invalid adapter id) and clear it. */
int bdlora_get_device_error(bdlora_pool_t pool, void* stream, int32_t* flag);

/* Adapter elements of one adapter of rank `rank` over the projections
 * `projs` (true rank, no padding): sum over projections and slices of
 * d_in*rank + rank*slice_out (the per-device factor shapes of Alg. 1/2).
 * Pure host function. */
int bdlora_adapter_elems(const bdlora_proj_desc* projs, int32_t n_projs, int32_t rank,
                         int64_t* elems);

/* Device memory a pool with these arguments would hold: adapter slabs
 * (every slot sized for max_rank, ranks padded to multiples of 8) and the
 * per-batch workspace (when max_tokens is above BDLORA_DECODE_MAX_T it
 * includes a fixed 64 MiB of fp32 partial tiles for the medium-batch base
 * product and the large-tile GEMM's split tiles, and 32 MiB for the split
 * shrink's partials).  Pure host function; validates the arguments as
 * bdlora_create_pool does (except the device). */
int bdlora_pool_size(const bdlora_proj_desc* projs, int32_t n_projs, int32_t max_slots,
                     int32_t max_rank, int32_t max_tokens, int64_t* slab_bytes,
                     int64_t* workspace_bytes);

/* Device bytes the pool holds (adapter slabs + workspace). */
int bdlora_pool_bytes(bdlora_pool_t pool, int64_t* bytes);

/* Timing hooks.  bdlora_profile_begin(pool, n) makes the next n forward
 * calls record HIP events around each of their launches on the caller's
 * stream, in four intervals: for a decode batch (BDLORA_PATH_DECODE) plan
 * and packing, K-split shrink and base partials, epilogue, nothing; for a
 * larger batch plan and packing, shrink, base product (with the fused
 * expand, or for BDLORA_PATH_MEDIUM the partials), and for
 * BDLORA_PATH_MEDIUM its epilogue (partials plus expand), else nothing.
 * bdlora_profile_end waits for them and writes the mean duration in
 * milliseconds of each interval to ms[0..3] (an empty interval reads about
 * 0) and the number of recorded calls to *n.  The calls averaged should
 * all take the same sequence. */
int bdlora_profile_begin(bdlora_pool_t pool, int32_t n);
int bdlora_profile_end(bdlora_pool_t pool, float* ms, int32_t* n);

/* Which launch sequence served the last forward call on this pool (known
 * when the call returns; the kernels may still be running), for tests and
 * tuning: *path = 0 before any forward, else one of
 *   BDLORA_PATH_DECODE  split-K decode launches (T <= BDLORA_DECODE_MAX_T)
 *   BDLORA_PATH_TILE64  64-row tiles, base product with the fused expand
 *   BDLORA_PATH_MEDIUM  all rows of the batch in one tile (bf16 weights,
 *                       T <= 256, layers whose weight is large against the
 *                       fp32 partials or batches of at most 8 tokens per
 *                       loaded adapter), then an epilogue that adds the
 *                       partials and the expand; the shrink runs beside the
 *                       base product on a stream the pool owns, forked from
 *                       the caller's stream after the plan and joined back
 *                       before the epilogue (graph capture follows the fork)
 *   BDLORA_PATH_LARGE   256 x 256 tiles (bf16 weights, T > 256)
 * INVALID_ARG for a null pool or path. */
#define BDLORA_PATH_DECODE 1
#define BDLORA_PATH_TILE64 2
#define BDLORA_PATH_MEDIUM 3
#define BDLORA_PATH_LARGE  4
int bdlora_last_path(bdlora_pool_t pool, int32_t* path);

/* Message of the last failing call on this thread ("" if none). */
const char* bdlora_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* BDLORA_H */
