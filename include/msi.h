/*
 * msi.h -- C ABI of the slot-backed routed-expert MoE layer for MI355X (gfx950).
 *
 * One MoE FFN layer (router softmax/top-K, token-by-expert permutation,
 * gate/up projections with SiLU gating, down projection, weighted combine plus
 * an always-on shared expert) executes against a bounded pool of reusable GPU
 * expert slots.  Logical expert objects live in caller-owned host windows; the
 * plan copies them into slots with stable device addresses, versions every
 * copy with a generation, and the compute kernels check the generation of
 * each slot they read, failing closed on a mismatch.
 *
 * The plan abstraction follows the paper's Design section: an immutable
 * manifest of objects, extents, windows and slots with stable addresses, and
 * replacement policy kept apart from the lifecycle ("A Shared Cross-Adapter
 * Plan Core"); slot generations and bundle publication ("Stable Slots and
 * Bundle Publication"); the separate window / GPU-slot state machines with
 * tickets, epochs and consumer counts ("Separate Window and GPU-Slot
 * Lifecycles"); and the scheduling loop of the Implementation section
 * ("Scheduling and copies": layer entry requests the bundle, misses are
 * copied into reserved slots, a device event publishes readiness, layer exit
 * releases the consumer ticket).  The lifetime row (L) of the paper's table
 * of certificate obligations is the error behaviour below.  The MoE
 * arithmetic itself is the layer every selected expert executes in the
 * paper's principal experiment ("Output-Exact Execution Beyond the
 * Full-Residency Envelope": the stock router, then the complete gate, up and
 * down projections).
 *
 * Conventions
 *  - Every call returns msi_status (0 = MSI_OK, negative = error).  The text
 *    of the last error on the calling thread is msi_last_error().  No C++
 *    exception crosses this boundary.
 *  - The caller owns every large buffer: the slot pool (device), the host
 *    windows (pinned host memory), x / out / routing arrays / workspace
 *    (device), and the HIP streams (passed as void* = hipStream_t; NULL is the
 *    null stream).  The plan owns host metadata and small device arrays
 *    (slot generation words, status word, schedule tables), freed by
 *    msi_plan_destroy.
 *  - Device pointers must be 16-byte aligned; the slot pool and slot stride
 *    256-byte aligned.
 *  - A plan is not thread-safe: calls on one plan must not overlap.  Plans
 *    on the same device are independent.
 *  - Storage formats (wdtype): MSI_W_F32 binary32; MSI_W_BF16 bfloat16 (top
 *    half of binary32); MSI_W_Q4B32 4-bit blocks: a [rows, cols] matrix is
 *    nibbles [rows, cols/2] (element 2j in the low nibble of byte j, 4-bit
 *    two's complement) followed by fp16 scales [rows, cols/32], value =
 *    scale * q.  MSI_W_KQ, the mixed super-block format of the quantized
 *    experts (the paper's 4.5 / 6.5625 bits-per-weight representation,
 *    Implementation section): Wg and Wu in k4 -- nibbles [rows, cols/2]
 *    (unsigned, element 2j in the low nibble of byte j) followed by a 16-byte
 *    header per (row, 256-element super-block): fp16 d, fp16 dmin, eight
 *    6-bit sub-block scales sc_j, eight 6-bit mins m_j (each group of eight a
 *    48-bit little-endian field, j-th at bits 6j); value = d sc_j q - dmin m_j
 *    for the j-th 32-element sub-block -- and Wd in k6: low nibbles
 *    [rows, cols/2], high 2-bit parts [rows, cols/4] (element 4j + t at bits
 *    2t of byte j), int8 scales [rows, cols/16], fp16 d [rows, cols/256];
 *    q = low | high << 4, value = d sc_j (q - 32) for the j-th 16-element
 *    sub-block.  KQ needs d_ff % 256 == 0.  Hidden states and the router
 *    weight are f32 for MSI_W_F32 and bf16 otherwise.
 *  - An expert object is [Wg | Wu | Wd]: Wg, Wu are [d_ff, d_model] and Wd is
 *    [d_model, d_ff], each row-major with the reduction axis contiguous.
 *    The router weight is [n_experts, d_model] row-major.
 */
#ifndef MSI_H
#define MSI_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MSI_ABI_VERSION 3u

typedef int32_t msi_status;

#define MSI_OK 0
#define MSI_E_INVALID_ARG (-1)  /* malformed argument, shape or alignment            */
#define MSI_E_SHORT (-2)        /* extent shorter/longer than the object, or past the window */
#define MSI_E_WRONG_OBJECT (-3) /* object not in this layer's manifest / slot not in its pool */
#define MSI_E_BUSY (-4)         /* slot has live consumers; no slot can be freed      */
#define MSI_E_STALE (-5)        /* a kernel saw a slot generation it did not expect    */
#define MSI_E_DEVICE (-6)       /* HIP runtime error                                  */
#define MSI_E_NOMEM (-7)        /* workspace too small or host allocation failed      */
#define MSI_E_STATE (-8)        /* lifecycle transition not allowed in this state     */
#define MSI_E_IO (-9)           /* a source read completed with a negative status (EIO...) */

typedef enum { MSI_W_F32 = 0, MSI_W_BF16 = 1, MSI_W_Q4B32 = 2, MSI_W_KQ = 3 } msi_wdtype;

typedef struct msi_plan msi_plan;

/* One logical object of the manifest: expert `expert` of layer `layer`,
 * stored as `nbytes` bytes at `offset` inside host window `window`. */
typedef struct {
    uint32_t layer;
    uint32_t expert;
    uint32_t window;
    uint32_t reserved;
    uint64_t offset;
    uint64_t nbytes;
} msi_object_desc;

/* Canonical source of expert objects (the bounded source service of the
 * Design section, "Bounded Source Service"): one extent of one object in a
 * canonical file.  An object is the concatenation of its extents in
 * component order (e.g. three components: Wg, Wu, Wd, read and checked
 * separately and published together as one bundle). */
typedef struct {
    uint32_t layer;
    uint32_t expert;
    uint32_t component;          /* 0, 1, ... without gaps, at most 4 per object */
    uint32_t file;               /* index into msi_source_desc.files             */
    uint64_t offset;             /* byte offset of the extent in the file        */
    uint64_t nbytes;             /* logical bytes                                */
} msi_extent_desc;

#define MSI_SOURCE_BUFFERED_OK 1u   /* read through the page cache where direct I/O is refused */

typedef struct {
    const char *const *files;    /* canonical files, read only                   */
    uint32_t n_files;
    uint32_t inflight;           /* reads in flight at most, 1..8                */
    uint32_t flags;              /* MSI_SOURCE_*                                 */
    uint32_t align;              /* direct-I/O block, power of two (0 -> 4096)   */
    const msi_extent_desc *extents;
    uint32_t n_extents;
    uint32_t reserved;
} msi_source_desc;

/* Immutable manifest ("A Shared Cross-Adapter Plan Core").  Slot s (0 <= s < pool_slots) of layer l
 * lives at slot_pool + (l * pool_slots + s) * slot_stride for the life of the
 * plan, where pool_slots = slots_per_layer, or transient_slots when
 * slots_per_layer == 0 (zero-cache: every use refills, nothing is retained
 * across rounds or calls).  slot_pool_bytes must cover
 * n_layers * pool_slots * slot_stride. */
typedef struct {
    uint32_t abi_version;        /* MSI_ABI_VERSION */
    uint32_t n_layers;
    uint32_t n_experts;          /* E, routed experts per layer, <= 1024     */
    uint32_t d_model;            /* d, multiple of 256                        */
    uint32_t d_ff;               /* I, expert intermediate, multiple of 128   */
    uint32_t top_k;              /* K, 1 <= K <= min(E, 16)                   */
    uint32_t wdtype;             /* msi_wdtype                                */
    uint32_t slots_per_layer;    /* C >= 0; 0 selects zero-cache              */
    uint32_t transient_slots;    /* zero-cache staging slots (0 -> 8), >= 2   */
    uint32_t policy;             /* msi_policy: replacement among demand slots */
    void *slot_pool;             /* device, caller-owned                      */
    uint64_t slot_pool_bytes;
    uint64_t slot_stride;        /* >= object bytes, multiple of 256          */
    const void *const *windows;  /* n_windows host pointers, caller-owned; pinned memory */
    uint32_t n_windows;
    uint32_t n_objects;
    uint64_t window_bytes;       /* size of every window                      */
    const msi_object_desc *objects;
    /* NULL: every object lives in a window (objects[]).  Otherwise objects
     * are read from canonical files (source->extents, n_objects must be 0)
     * and the windows are the source's staging windows: n_windows buffers of
     * window_bytes (a multiple of source->align) aligned to source->align,
     * each holding one object's covering reads while it is read and then
     * copied to its slot (states Free -> Reading -> HostReady -> Copying ->
     * Free), so the source holds at most n_windows * window_bytes. */
    const msi_source_desc *source;
    /* Two-bank prefetch: the last prefetch_slots slots of each layer's pool
     * form its prefetch bank, filled only by msi_prefetch; demand misses of a
     * forward go to the other slots (the demand bank), so a wrong prefetch
     * never evicts a cached object.  0 (no bank) or < slots_per_layer; 0 for
     * zero-cache plans. */
    uint32_t prefetch_slots;
    uint32_t reserved1;
} msi_plan_desc;

/* Replacement policies (kept apart from the slot lifecycle: "A Shared
 * Cross-Adapter Plan Core").  LRU: the least recently used slot without
 * consumers.  PROTECTED_LRU: a segmented LRU -- a hit moves the object into
 * a protected segment of at most half the demand bank (its least recently
 * used member drops back when it overflows); victims are the least recently
 * used unprotected slots first, protected ones only when no other is
 * left. */
typedef enum { MSI_POLICY_LRU = 0, MSI_POLICY_PROTECTED_LRU = 1 } msi_policy;

/* Ticket of a fill ("Separate Window and GPU-Slot Lifecycles": tickets carry object, generation, epoch and
 * resource identity). */
typedef struct {
    uint32_t layer;
    uint32_t expert;
    int32_t slot;
    uint32_t generation;
    uint32_t epoch;
    uint32_t hit;                /* 1 if the object was already resident       */
} msi_ticket;

/* Device arrays describing one routing of T tokens (all caller-owned).  For
 * an empty batch (T == 0) the per-row arrays may be null; counts, offsets and
 * demand are always written (all zero for T == 0). */
typedef struct {
    int32_t *idx;                /* [T, K] selected experts, ascending per token      */
    float *weights;              /* [T, K] gate weights (restricted softmax), fp32    */
    int32_t *counts;             /* [E] tokens per expert                             */
    int32_t *offsets;            /* [E + 1] exclusive prefix of counts                */
    int32_t *demand;             /* [E + 1] demanded experts: their number, then their ids ascending */
    int32_t *perm;               /* [T * K] token of each permuted row; rows ordered by (expert, token) */
    int32_t *inv;                /* [T, K] permuted row of each (token, k)            */
    float *row_weight;           /* [T * K] gate weight of each permuted row          */
} msi_routing;

typedef struct {
    uint32_t n_tokens;           /* T >= 0                                             */
    uint32_t reserved;
    const void *x;               /* [T, d] hidden states (f32 or bf16, see wdtype)     */
    const void *w_router;        /* [E, d] router weight, same type as x               */
    const float *bias;           /* [E] added to the logits before selection, or NULL  */
    msi_routing r;               /* outputs                                            */
    void *workspace;             /* msi_workspace_size(plan, T) bytes                  */
    uint64_t workspace_bytes;
} msi_route_args;

typedef struct {
    uint32_t layer;
    uint32_t n_tokens;           /* T, same as the routing's                           */
    const void *x;               /* [T, d] the routed hidden states                    */
    msi_routing r;               /* produced by msi_route for this x                    */
    const void *shared_object;   /* device [Wg | Wu | Wd] of the always-on shared expert, or NULL */
    float *out;                  /* [T, d] fp32 output; written only on MSI_OK         */
    void *workspace;
    uint64_t workspace_bytes;
} msi_forward_args;

/* Per-slot view for tests and telemetry. */
typedef enum {
    MSI_SLOT_VACANT = 0,
    MSI_SLOT_LOADING = 1,
    MSI_SLOT_DEVICE_READY = 2,
    MSI_SLOT_IN_USE = 3,
    MSI_SLOT_RECYCLABLE = 4
} msi_slot_state;

typedef struct {
    uint32_t state;              /* msi_slot_state                                     */
    int32_t expert;              /* resident object, -1 if none                         */
    uint32_t generation;
    uint32_t epoch;
    uint32_t consumers;          /* live consumers (forward rounds + holds)             */
    uint32_t holds;              /* consumers held through msi_slot_hold                */
    uint64_t last_use;           /* LRU tick                                            */
} msi_slot_info;

typedef struct {
    uint64_t forwards;
    uint64_t rounds;
    uint64_t fills;              /* copies submitted                                    */
    uint64_t fills_published;    /* completions that became DeviceReady                 */
    uint64_t fills_discarded;    /* completions rejected (epoch/generation mismatch)    */
    uint64_t hits;               /* demanded objects found resident                     */
    uint64_t misses;
    uint64_t evictions;          /* resident objects replaced                           */
    uint64_t h2d_bytes;
    uint64_t rejections;         /* BUSY / WRONG_OBJECT / SHORT / STATE returned        */
    uint64_t stale_detected;     /* forwards that returned MSI_E_STALE                  */
    uint64_t fills_in_flight;
    uint64_t windows_busy;       /* windows with a copy in flight                       */
    uint64_t consumers_live;
    uint32_t epoch;
    uint32_t reserved;
    uint64_t prefetch_fills;     /* fills issued by msi_prefetch                         */
    uint64_t prefetch_used;      /* prefetched objects a forward then used               */
} msi_stats;

/* Kernel kinds of the per-kind timing telemetry. */
typedef enum {
    MSI_K_ROUTER_LOGITS = 0,
    MSI_K_TOPK = 1,
    MSI_K_PERMUTE = 2,
    MSI_K_GATEUP_TILE = 3,     /* routed experts, tiled MFMA path                 */
    MSI_K_GATEUP_STREAM = 4,   /* routed experts, weight-streaming path           */
    MSI_K_DOWN_TILE = 5,
    MSI_K_DOWN_STREAM = 6,
    MSI_K_EXPERT_F32 = 7,      /* fp32 layers, gate/up and down                   */
    MSI_K_SHARED = 8,          /* shared expert, gate/up and down                 */
    MSI_K_COMBINE = 9,
    MSI_K_FILL = 10,           /* one batch of slot fills on the side stream      */
    MSI_NKERN = 11
} msi_kernel_kind;

typedef struct {
    uint64_t launches[MSI_NKERN];
    double ms[MSI_NKERN];       /* summed device time between events around each launch */
} msi_timings;

/* Text of the last error on this thread ("" if none).  Never NULL. */
const char *msi_last_error(void);

/* ABI version of the loaded library (MSI_ABI_VERSION). */
uint32_t msi_abi_version(void);

/* Validate the manifest and create a plan on the current HIP device
 * ("A Shared Cross-Adapter Plan Core"; stable addresses, "Stable Slots and
 * Bundle Publication"; extent rejection conditions, "Bounded Source
 * Service").  Errors: MSI_E_INVALID_ARG (shape, alignment, pool too small,
 * duplicate (layer, expert), window index out of range), MSI_E_SHORT (extent
 * past its window, or nbytes != object size for wdtype and shape),
 * MSI_E_DEVICE.  With a source: MSI_E_INVALID_ARG (a file that cannot be
 * opened, component gaps or duplicates, misaligned or too small windows,
 * in-flight limit outside 1..8), MSI_E_SHORT (an extent past its file's end,
 * or an object whose extents do not add up to the object size).  All slots
 * start Vacant with generation 0, epoch 0. */
msi_status msi_plan_create(const msi_plan_desc *desc, msi_plan **out);

/* Drain in-flight fills (and every submitted source read) and free
 * plan-owned memory.  MSI_E_BUSY (plan kept)
 * if a consumer is still held through msi_slot_hold (shutdown with a live
 * consumer: "Separate Window and GPU-Slot Lifecycles" and the fault-mode
 * table of "Integrated Deterministic Faults"). */
msi_status msi_plan_destroy(msi_plan *plan);

/* Advance the request epoch ("Separate Window and GPU-Slot Lifecycles").
 * Fills still in flight, including source reads, become unpublishable: their
 * completion leaves the slot Vacant (a read completing later frees its
 * window without any copy).  Resident DeviceReady slots stay valid.
 * MSI_E_BUSY if a consumer is held. */
msi_status msi_plan_reset(msi_plan *plan);

/* Bytes of device workspace msi_route and msi_moe_forward need for T tokens.
 * Layout (each part starts on a 256-byte boundary; ab = 4 for MSI_W_F32,
 * else 2): router logits [T, E] f32 | per-block expert histograms
 * [ceil(T / 256), E] i32 | act [T * K, d_ff] (permuted rows) | shared-expert
 * act [T, d_ff] | y [T * K, d_model] (weighted expert outputs, permuted
 * rows) | shared-expert output [T, d_model]; act, y and their shared parts
 * in ab-byte elements (bf16 or f32).  Contents are scratch between calls. */
msi_status msi_workspace_size(const msi_plan *plan, uint32_t n_tokens, uint64_t *bytes);

/* Make expert `expert` of `layer` resident ("Stable Slots and Bundle
 * Publication"; Implementation, "Scheduling and copies").
 * slot = -1 lets the replacement policy choose (least recently used slot
 * without consumers); slot >= 0 forces that slot.  If the object is already
 * resident and ready (in `slot` when forced) this is a hit: the ticket
 * carries the current generation and nothing is copied.  Otherwise the slot
 * goes Loading with generation g+1 and, on `side_stream`, its device
 * generation word is invalidated, the extent is copied window -> slot, the
 * word is set to g+1 and a ready event is recorded.  The completion is
 * published (DeviceReady) only if the ticket's epoch and generation are still
 * current when it is observed.  Errors: MSI_E_WRONG_OBJECT (no such object in
 * this layer's manifest, or slot outside the layer's pool), MSI_E_BUSY (forced
 * slot has live consumers, or every slot does), MSI_E_DEVICE. */
msi_status msi_slot_fill(msi_plan *plan, uint32_t layer, uint32_t expert, int32_t slot,
                         void *side_stream, msi_ticket *ticket);

/* Next-layer prefetch into the layer's prefetch bank (two-bank prefetch,
 * the mechanism the paper's Qwen natural-utility experiment runs beside its
 * protected LRU): for each of the n listed experts (host array) that is not
 * already resident or loading, fill it into the least recently used
 * prefetch-bank slot without consumers, asynchronously on side_stream (or
 * through the source), at most prefetch_slots fills per call; *issued (may
 * be NULL) receives the number of fills.  A later forward finds prefetched
 * objects as hits.  Errors: MSI_E_INVALID_ARG (no prefetch bank, layer out
 * of range), MSI_E_WRONG_OBJECT (an expert outside the layer's manifest),
 * MSI_E_DEVICE. */
msi_status msi_prefetch(msi_plan *plan, uint32_t layer, const int32_t *experts, uint32_t n, void *side_stream,
                        uint32_t *issued);

/* Observe completed fills and consumer releases without blocking. */
msi_status msi_plan_poll(msi_plan *plan);

/* Router and permutation on `stream` (no host synchronisation): logits
 * (bf16 MFMA or fp32 with fp32 accumulation) plus bias, top-K by (logit desc,
 * expert id asc), softmax restricted to the selected set in fp32, then the
 * stable token-by-expert permutation and the list of demanded experts.  Fully
 * deterministic.  For 1 <= T <= 16 bf16 tokens all of it is one launch whose
 * workgroups count their arrival in a plan-owned word: msi_route calls on one
 * plan must not overlap in time (e.g. on two streams without ordering).
 * Errors: MSI_E_INVALID_ARG, MSI_E_NOMEM (workspace), MSI_E_DEVICE. */
msi_status msi_route(msi_plan *plan, const msi_route_args *args, void *stream);

/* One MoE layer against the slot pool (Implementation, "Scheduling and
 * copies").  Reads the
 * per-expert counts (one device-to-host copy), resolves the demanded set
 * against the residency state (hits first, then misses in ascending expert
 * id, in rounds of at most the pool size), fills misses on `side_stream`
 * overlapped with compute, runs the expert kernels on `compute_stream` with
 * in-kernel generation checks, runs the shared expert, and publishes
 * out[t] = shared(x_t) + sum over the token's experts in ascending id of
 * w * expert(x_t), in fp32.  Blocks until the status word is known.
 * When the layer's previous forward needed no fill and T is within the stream
 * path, the work list is instead built on the device from r.demand and the
 * published residency table (no host round trip before the expert kernels),
 * and the call returns once the combine has published the status: output rows
 * may still be in flight, ordered before later work on `compute_stream`.
 * out is bit-identical for every slot capacity.  Errors: MSI_E_STALE (a
 * kernel saw an unexpected slot generation; out is untouched), MSI_E_BUSY (no
 * slot could be freed), MSI_E_INVALID_ARG, MSI_E_NOMEM, MSI_E_DEVICE. */
msi_status msi_moe_forward(msi_plan *plan, const msi_forward_args *args,
                           void *compute_stream, void *side_stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same
 * forward as msi_moe_forward, with the same result, but its act / y scratch
 * (the workspace parts after the histograms, see msi_workspace_size) is a
 * static device array of the library, MSI_NOALLOC_SCRATCH_BYTES per device,
 * held from the library's load until the process ends.  args->workspace must
 * be NULL and args->workspace_bytes 0.  It calls no hipMalloc / hipFree and
 * no allocating library routine.  Every call on one device shares that
 * device's array and leaves its contents behind (nothing in it needs to
 * start zeroed: a forward writes every row it reads), so calls that overlap
 * on one device race: order them on one stream or serialise them.  Errors:
 * those of msi_moe_forward; MSI_E_INVALID_ARG when T tokens need more than
 * MSI_NOALLOC_SCRATCH_BYTES (T * (K + 1) * (d_ff + d_model) * 2 bytes plus
 * alignment for bf16 / 4-bit layers: about 1,190 tokens at d_model 2048,
 * d_ff 512, K 10) or a workspace is passed. */
#define MSI_NOALLOC_SCRATCH_BYTES (64u << 20)
msi_status msi_moe_forward_noalloc(msi_plan *plan, const msi_forward_args *args, void *compute_stream,
                                   void *side_stream);

/* Hold / release one external consumer on a slot (a consumer ticket that
 * outlives a forward; a held slot is never chosen as a victim and cannot be
 * refilled).  MSI_E_STATE when unholding a slot with no holds. */
msi_status msi_slot_hold(msi_plan *plan, uint32_t layer, uint32_t slot);
msi_status msi_slot_unhold(msi_plan *plan, uint32_t layer, uint32_t slot);

msi_status msi_slot_query(const msi_plan *plan, uint32_t layer, uint32_t slot, msi_slot_info *info);
msi_status msi_plan_stats(const msi_plan *plan, msi_stats *stats);

/* Telemetry: enable = 0 off, 1 every kernel kind, otherwise a bit mask of
 * (1 << msi_kernel_kind).  Each selected kernel launch of route/forward on
 * this plan carries two HIP events that the runtime records at the start of
 * its first kernel and the end of its last kernel; a fill (a copy) is
 * bracketed by two events on the side stream.  msi_plan_timings waits for
 * the recorded events, accumulates the elapsed times per kernel kind into
 * *out and, if reset != 0, clears the accumulators.
 * msi_plan_set_timing_period: time only every period-th launch of each kind
 * (period >= 1, default 1), to keep the per-launch event cost off most
 * launches; MSI_E_INVALID_ARG for period 0. */
msi_status msi_plan_set_timing(msi_plan *plan, int enable);
msi_status msi_plan_set_timing_period(msi_plan *plan, uint32_t period);
msi_status msi_plan_timings(msi_plan *plan, msi_timings *out, int reset);

/* Residual stream between stacked layers (attention omitted), row-major
 * [rows, cols]: msi_residual_init sets h = float(x0); msi_residual_add does
 * h += out.  Both then write the next layer's input x = bf16_rne(h / rms(h))
 * per row, rms(h) = sqrt(mean(h^2) + 1e-6) summed in fp32 in a fixed order
 * (an unweighted RMSNorm, as a transformer block normalizes its input; without
 * it the gated FFN's quadratic response overflows a deep stack).  x0 and x
 * may alias.  Device pointers, on `stream`. */
msi_status msi_residual_init(const uint16_t *x0_bf16, float *h, uint16_t *x_bf16, uint32_t rows, uint32_t cols,
                             void *stream);
msi_status msi_residual_add(const float *out, float *h, uint16_t *x_bf16, uint32_t rows, uint32_t cols,
                            void *stream);

/* Source-service counters (plans with a source; zeros otherwise). */
typedef struct {
    uint64_t reads_issued, reads_completed, reads_failed;
    uint64_t requests, requests_ready, requests_failed, requests_stale;
    uint64_t logical_bytes, physical_bytes, padding_bytes;   /* physical: aligned covering reads */
    uint64_t peak_depth;         /* most reads in flight at once                       */
    uint64_t windows_busy;       /* staging windows not Free now                       */
    double read_seconds;         /* summed latency of the reads                        */
    double wait_seconds;         /* time forwards spent blocked on the source          */
    uint32_t direct_files;       /* files read with direct I/O                         */
    uint32_t buffered_files;     /* files read through the page cache (fallback)       */
    uint64_t bounced_reads;      /* direct reads staged through a 4 MiB bounce buffer per I/O
                                    worker because the windows' pages refuse direct reads */
} msi_source_stats;
msi_status msi_source_stats_get(const msi_plan *plan, msi_source_stats *stats);

/* Test hooks of the source's rejection conditions: the next read of extent
 * `component` of (layer, expert) returns short (MSI_FAULT_SHORT), fails with
 * EIO (MSI_FAULT_EIO) or is held until msi_debug_source_release
 * (MSI_FAULT_HOLD; a held read completes by itself after 30 s).  The request
 * then fails closed: its window returns to Free, no copy is made and nothing
 * is published; a forward that needed it returns MSI_E_SHORT / MSI_E_IO with
 * out untouched. */
#define MSI_FAULT_SHORT 1u
#define MSI_FAULT_EIO 2u
#define MSI_FAULT_HOLD 3u
msi_status msi_debug_source_fault(msi_plan *plan, uint32_t layer, uint32_t expert, uint32_t component,
                                  uint32_t mode);
msi_status msi_debug_source_release(msi_plan *plan);

/* Test hook: overwrite one slot's device generation word (synchronously). */
msi_status msi_debug_set_device_gen(msi_plan *plan, uint32_t layer, uint32_t slot, uint32_t gen);

/* Expert-path selector of a forward, for tests: tokens-per-expert at or below
 * which the weight-streaming path runs (the rest take the tiled MFMA path).
 * Returns the current value; 0 keeps it.  The choice is a function of the
 * routing only, never of capacity. */
uint32_t msi_stream_threshold(uint32_t new_value);

#ifdef __cplusplus
}
#endif

#endif /* MSI_H */
