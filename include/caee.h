/*
 * caee.h -- C ABI of the Cost-Aware Expert Execution (CAEE) MoE-layer
 * library for AMD Instinct MI355X (gfx950).
 *
 * One MoE layer per call, following "Beyond Uniform Experts: Cost-Aware
 * Expert Execution for Efficient Multi-Device MoE Inference" (arxiv
 * 2606.29982):
 *   1. router scores and group-limited top-k K_t per token (Sec. II-A);
 *   2. cost-aware pruning of the activated set A_act into A_trans:
 *      importance threshold, baseline cost F_base as the maximum over bins
 *      (devices) of the summed expert cost, cost-invariant expansion
 *      (Sec. IV-A cost model, Sec. IV-B steps 1-4);
 *   3. compensation: pruned experts are masked and each token's freed slots
 *      are re-filled from A_trans (Sec. IV-C), weights renormalised;
 *   4. the surviving experts (plus shared experts) run as a grouped SwiGLU
 *      FFN and their outputs are combined with the gate weights (the MoE
 *      output equation of Sec. II-A).
 *
 * Conventions shared by every entry point
 *   - Every tensor pointer is caller-owned DEVICE memory (hipMalloc'd or a
 *     torch CUDA tensor), row-major and densely packed, 16-byte aligned.
 *     Sizes are in elements unless stated.  The library allocates no device
 *     memory: scratch space comes from the caller's workspace `ws`.
 *   - Calls are asynchronous on `stream` (a hipStream_t; NULL = the null
 *     stream).  Inputs must stay valid and unmodified, and outputs must not
 *     be read, until the stream has reached the end of the call.
 *   - All arguments are validated on the host before anything is launched.
 *     On any error nothing is launched, outputs are untouched, and
 *     caee_last_error() returns a message for the calling thread.
 *   - Device contents cannot be checked on the host.  Preconditions that
 *     the caller must guarantee: logits, bias and costs are finite; costs
 *     are >= 0; bin[e] is in [0, n_bins).  Violations give unspecified
 *     (but memory-safe) results.
 *   - Decisions (selection, importance threshold, cost comparisons) are
 *     computed in float64, ties going to the lower expert or group index,
 *     so results are deterministic and independent of launch shape.
 *     Per-bin cost sums are exact (hence independent of summation order)
 *     while, within each bin, the nonzero costs span less than 2^20
 *     (largest / smallest); beyond that range they may differ from an
 *     ascending-order sum in the last bit.
 */
#ifndef CAEE_H
#define CAEE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define CAEE_ABI_VERSION 8

typedef enum caee_status {
    CAEE_OK = 0,
    CAEE_ERR_INVALID_ARG = 1,  /* bad descriptor field, NULL or misaligned pointer */
    CAEE_ERR_UNSUPPORTED = 2,  /* well-formed but outside this build's limits */
    CAEE_ERR_WORKSPACE = 3,    /* ws NULL or ws_bytes < caee_workspace_size() */
    CAEE_ERR_HIP = 4,          /* a HIP runtime call or a kernel launch failed */
    CAEE_ERR_CAPACITY = 5      /* an offload call needs more device slots than it was given */
} caee_status_t;

typedef enum caee_dtype {
    CAEE_F32 = 0,       /* IEEE binary32 */
    CAEE_BF16 = 1,      /* bfloat16 */
    CAEE_FP8_E4M3 = 2   /* OCP FP8 E4M3 (max 448), used with fp32 block scales */
} caee_dtype_t;

/* Mandatory-set rule of the pruning step (Sec. IV-B step 1).  A_must holds
 * exactly the experts the rule makes mandatory.  The paper's steps leave one
 * case undefined: when steps 1-4 leave A_trans empty (no mandatory expert and
 * no candidate the expansion keeps), the final top-k of Sec. IV-C has nothing
 * to choose from.  Only then are steps 2-4 run again with every token's own
 * top expert (largest G, lower index on ties) added to A_must; stats[8]
 * reports it.  desc.keep_top1 = 1 adds those experts in every call. */
typedef enum caee_importance {
    /* I(e) = largest normalised gate weight any token of the batch gives e;
     * A_must = {e : I(e) >= tau}.  Sec. IV-B leaves I(e) open; with this
     * choice no (token, expert) pair whose gate weight reaches tau is pruned. */
    CAEE_IMPORTANCE_MAX = 0,
    /* I(e) = sum over tokens of G(t)_e, the on-device rule of Sec. V-C;
     * A_must = {e : I(e) >= tau}.  Candidates are visited by this sum. */
    CAEE_IMPORTANCE_SUM = 1,
    /* Cumulative importance ratio, the offloading rule of Sec. V-B: each
     * token keeps its shortest prefix of experts (gate weight descending)
     * whose share of the token's gate mass reaches tau (theta_imp); A_must
     * is the union.  Candidates are visited by their largest gate weight. */
    CAEE_IMPORTANCE_CIR = 2
} caee_importance_t;

/* How compensation (Sec. IV-C) fills the slots pruning freed in a token's
 * list.  SCORE is the paper's mechanism; NONE and RANDOM exist for its
 * ablation (random selection among the executed experts vs the proposed
 * compensation); LITERAL is the other reading of its top-k step. */
typedef enum caee_refill {
    /* Best router keys of A_trans minus K_t (no group limit). */
    CAEE_REFILL_SCORE = 0,
    /* No refill: K_final = K_t within A_trans, weights renormalised over it. */
    CAEE_REFILL_NONE = 1,
    /* The experts of A_trans minus K_t with the largest random keys: the top
     * 53 bits of the SplitMix64 output for counter (seed << 32) | (t*E + e),
     * t the token's index in the call; ties to the lower index. */
    CAEE_REFILL_RANDOM = 2,
    /* Sec. IV-C's top-k of the masked scores taken literally: K_final = the
     * k best router keys of A_trans (ties to the lower index), whether or
     * not they were in K_t, no group limit.  May drop a token's own
     * surviving expert; not the plain layer at tau = 0 in general. */
    CAEE_REFILL_LITERAL = 3
} caee_refill_t;

/* Shape and hyper-parameters of one MoE layer call. */
typedef struct caee_layer_desc {
    int32_t T;            /* tokens in the batch, >= 0 (0: the call does nothing) */
    int32_t d;            /* hidden size, multiple of 128 */
    int32_t f;            /* expert intermediate size, multiple of 128 */
    int32_t E;            /* routed experts, 1..256 */
    int32_t n_group;      /* expert groups (group g = experts [g*E/n_group, (g+1)*E/n_group)) */
    int32_t topk_group;   /* groups kept per token, 1..n_group */
    int32_t k;            /* experts per token, 1..16 and <= topk_group*E/n_group */
    int32_t n_shared;     /* shared experts added to every token with weight 1, 0..4 */
    float routed_scaling; /* factor on the renormalised routed weights, finite and > 0 */
    float tau;            /* threshold of the importance rule (theta, or theta_imp for CIR), finite and >= 0;
                             0 disables pruning for MAX and SUM */
    int32_t n_bins;       /* devices/links of the max-aggregated layer cost (Sec. IV-A), 1..256 */
    int32_t importance;   /* caee_importance_t */
    int32_t x_dtype;      /* hidden-state dtype: CAEE_F32 with f32 weights, else CAEE_BF16 */
    int32_t w_dtype;      /* expert weight dtype: CAEE_F32, CAEE_BF16 or CAEE_FP8_E4M3 */
    int32_t y_dtype;      /* output dtype: CAEE_F32 or CAEE_BF16 */
    int32_t refill;       /* a caee_refill_t; CAEE_REFILL_SCORE is the paper's method */
    uint32_t seed;        /* CAEE_REFILL_RANDOM: seed of the random keys; ignored otherwise */
    int32_t keep_top1;    /* 0: A_must as Sec. IV-B step 1 defines it (the paper's method);
                             1: each token's own top expert is also mandatory in every call */
} caee_layer_desc_t;

/* Storage order of the expert matrices. */
typedef enum caee_layout {
    /* Row-major: matrix [R][K], K contiguous. */
    CAEE_LAYOUT_ROWMAJOR = 0,
    /* Tiled, the order the FFN kernels stream: for row tile t (rows
     * 16t..16t+15) and contraction step s (64 bytes of each row), one
     * 1024-byte block whose 16-byte piece j (j = r + 16*q, r < 16, q < 4)
     * is bytes [64s + 16q, 64s + 16q + 16) of row 16t + r; blocks ordered
     * by t, then s.  Same bytes as row-major, permuted; produced by
     * caee_pack_matrix. */
    CAEE_LAYOUT_TILED = 1
} caee_layout_t;

/* Expert weights.  Expert e's gate and up matrices are stacked as
 * w13[e] = [W1; W3] of shape [2f][d], its down matrix is w2[e] of shape
 * [d][f]; both K-contiguous (each row is one output feature).  The expert
 * computes W2 (silu(W1 x) * (W3 x)).
 * FP8: w13/w2 hold E4M3 codes and *_scale hold one fp32 scale per 128x128
 * block, w13_scale [E][2f/128][d/128] and w2_scale [E][d/128][f/128]; the
 * weight is code * scale.  *_scale must be NULL for other dtypes.
 * The shared experts use the same layout with n_shared in place of E.
 * `layout` applies to all four matrices (scales are always row-major). */
typedef struct caee_expert_weights {
    const void* w13;            /* [E][2f][d] */
    const void* w2;             /* [E][d][f] */
    const float* w13_scale;     /* FP8 only */
    const float* w2_scale;      /* FP8 only */
    const void* sh_w13;         /* [n_shared][2f][d], NULL iff n_shared == 0 */
    const void* sh_w2;          /* [n_shared][d][f] */
    const float* sh_w13_scale;  /* FP8 only */
    const float* sh_w2_scale;   /* FP8 only */
    int32_t layout;             /* caee_layout_t */
} caee_expert_weights_t;

/* Routing results, all caller-owned device memory.  Lists are in rank order
 * (router key s+bias descending, expert index ascending). */
typedef struct caee_route_out {
    int32_t* topk_ids;   /* [T][k] K_final after compensation; -1 in unused slots (required) */
    float* topk_w;       /* [T][k] routed_scaling * s_e / sum_{K_final} s; 0 in unused slots (required) */
    int32_t* orig_ids;   /* [T][k] K_t before pruning (optional, may be NULL) */
    uint32_t* masks;     /* [4][ceil(E/32)] bitmaps A_act, A_must, A_trans, pruned; bit e%32 of word e/32 (optional) */
    int32_t* stats;      /* [9] |A_act|, |A_must|, |A_cand|, promoted, pruned, |A_trans|,
                            refilled slots, empty slots, and 1 if A_trans came out empty and
                            each token's top expert was made mandatory, else 0 (optional) */
    double* bin_loads;   /* [3][n_bins] per-bin summed cost of A_act, of A_must (max = F_base)
                            and of A_trans (optional) */
} caee_route_out_t;

/* Bytes of workspace the three compute entry points need for `desc`
 * (the same value serves all three).  Host-only, launches nothing. */
caee_status_t caee_workspace_size(const caee_layer_desc_t* desc, size_t* bytes);

/* Routing, cost-aware pruning and compensation (Sec. II-A, IV-B, IV-C).
 *   logits [T][E] fp32 router logits; bias [E] fp32 selection bias or NULL;
 *   cost [E] fp32 per-expert cost R(e)*C(e) of Sec. IV-A (0 = resident);
 *   bin [E] int32 bin of each expert, NULL = all experts in bin 0
 *   (then n_bins must be 1).
 * Writes `out`.  `ws` must hold caee_workspace_size() bytes. */
caee_status_t caee_route_prune(const caee_layer_desc_t* desc, const float* logits,
                               const float* bias, const float* cost, const int32_t* bin,
                               const caee_route_out_t* out, void* ws, size_t ws_bytes,
                               void* stream);

/* Grouped SwiGLU expert FFN and weighted combine (Sec. II-A output
 * equation): y_t = sum_j topk_w[t][j] * E_{topk_ids[t][j]}(x_t) + sum_s E^sh_s(x_t).
 *   x [T][d] (x_dtype); topk_ids/topk_w [T][k] as written by
 *   caee_route_prune (an id outside [0,E) marks an empty slot and its
 *   weight is ignored; an expert named in several slots of one token adds
 *   its output once per slot, with that slot's weight); y [T][d] (y_dtype),
 *   fully overwritten. */
caee_status_t caee_expert_ffn(const caee_layer_desc_t* desc, const void* x,
                              const int32_t* topk_ids, const float* topk_w,
                              const caee_expert_weights_t* weights, void* y,
                              void* ws, size_t ws_bytes, void* stream);

/* The whole layer: caee_route_prune followed by caee_expert_ffn, without
 * leaving the device.  `out` may be NULL (routing results then live in the
 * workspace only); if given, it is filled as by caee_route_prune. */
caee_status_t caee_moe_layer(const caee_layer_desc_t* desc, const void* x,
                             const float* logits, const float* bias, const float* cost,
                             const int32_t* bin, const caee_expert_weights_t* weights,
                             void* y, const caee_route_out_t* out, void* ws,
                             size_t ws_bytes, void* stream);

/* Bytes of the library's own scratch array (per GPU) behind
 * caee_moe_layer_noalloc: enough for a DeepSeek-R1-shaped layer (d 7168,
 * f 2048, 256 experts, top-8, one shared expert) up to 128 tokens. */
#define CAEE_SCRATCH_BYTES (48u << 20)

/* caee_moe_layer without a caller workspace, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc).  Same arguments, results and
 * kernels as caee_moe_layer, minus ws/ws_bytes: the scratch space is a
 * file-scope device array of CAEE_SCRATCH_BYTES in the library, one per GPU,
 * whose address is looked up once per device on the first call there (with
 * that device current) and held until the process ends.  All kernels run on
 * `stream` (no second stream is created).  The call allocates nothing and
 * needs nothing in the array cleared: every byte the kernels read is written
 * earlier in the same call.
 * Returns CAEE_ERR_UNSUPPORTED, launching nothing, when the call needs more
 * than CAEE_SCRATCH_BYTES (caee_workspace_size tells).  Every call on one GPU
 * uses the same array: calls that overlap on one GPU (different streams or
 * threads without ordering between them) race and give undefined results. */
caee_status_t caee_moe_layer_noalloc(const caee_layer_desc_t* desc, const void* x,
                                     const float* logits, const float* bias, const float* cost,
                                     const int32_t* bin, const caee_expert_weights_t* weights,
                                     void* y, const caee_route_out_t* out, void* stream);

/* Repack `count` consecutive row-major matrices [rows][cols] of dtype
 * `w_dtype` from `src` into CAEE_LAYOUT_TILED order at `dst` (same size,
 * must not overlap).  rows must be a multiple of 16 and a row a multiple of
 * 64 bytes.  Asynchronous on `stream`; a one-time step when weights are
 * loaded (weights are static during inference).  Tiled weights let each
 * FFN wavefront stream one contiguous region instead of 32 rows, which is
 * what keeps HBM near its streaming bandwidth. */
caee_status_t caee_pack_matrix(int32_t w_dtype, const void* src, void* dst, int64_t rows, int64_t cols,
                               int64_t count, void* stream);

/* The activation quantiser of the 8-bit path: `rows` rows of `cols` values
 * (src_dtype CAEE_BF16 or CAEE_F32) to OCP E4M3 per row per 128 columns.
 * In fp32: scale = amax / 448 (1 for an all-zero block), code = value / scale
 * rounded to the nearest E4M3 value, ties to the even code, saturating at
 * 448.  q [rows][cols] uint8 codes, scale [rows][cols/128] fp32; cols must be
 * a multiple of 128.  Asynchronous on `stream`. */
caee_status_t caee_quantize_rows(int32_t src_dtype, const void* src, int64_t rows, int64_t cols, uint8_t* q,
                                 float* scale, void* stream);

/* ---------------------------------------------------------------------------
 * Offload residency.
 *
 * In the offloading deployment (Sec. V-B) every routed expert lives in host
 * memory and only some of them in device memory; an expert that is needed
 * but absent costs a host-to-device transfer of its S_e bytes over a link of
 * bandwidth B (the cost model of Sec. IV-A, where R(e,d) = 1 for such a miss
 * and 0 for a resident expert).  A caee_offload_t holds the residency state
 * of one layer: which expert each device cache slot holds and the last call
 * that used it.  Each caee_offload_layer call
 *   1. writes the cost table: 0 for a resident expert, `miss_cost` for the
 *      others, all experts in one bin (the host link), and runs routing,
 *      pruning and compensation with it on `stream` -- so pruning keeps the
 *      mandatory experts, promotes the resident candidates, and prunes the
 *      candidates that would have to be fetched;
 *   2. waits on the host for that routing step to finish (the only host
 *      synchronisation of the call) and reads A_trans;
 *   3. plans the call (caee_lru_step): experts of A_trans already resident
 *      are hits; the others are misses and go, in ascending expert order,
 *      into empty cache slots, then into the slots of the least recently
 *      used experts that this call does not need; once none is left, into
 *      the staging slots, which cache nothing;
 *   4. copies the misses host -> device with hipMemcpyAsync on
 *      `copy_stream`, `fetch_batch` experts at a time, while `stream` runs
 *      the FFN of the hits and shared experts and then of each batch once it
 *      has landed; a staging slot is refilled only after the FFN that read
 *      it has finished;
 *   5. combines all expert outputs into y on `stream`.
 * The result equals caee_moe_layer with the same cost table and weights.
 *
 * Ownership: host weights, device slots, shared weights, inputs, outputs and
 * the workspace are the caller's.  The handle allocates a few KB of device
 * and page-locked host memory for its tables and some HIP events, all freed
 * by caee_offload_destroy.  A handle is not thread-safe; calls on one
 * handle must come from one thread, in order. */
typedef struct caee_offload caee_offload_t;

typedef struct caee_offload_desc {
    /* Routed experts in host memory: host_w13[e] and host_w2[e] point to
     * expert e's matrices ([2f][d] and [d][f], in `layout` order), each in
     * page-locked memory (hipHostMalloc or a pinned torch tensor) so that
     * copies run asynchronously. */
    const void* const* host_w13;   /* host array of E pointers */
    const void* const* host_w2;    /* host array of E pointers */
    /* Device slots: slot i holds one expert at slot_w13 + i*(2f*d) elements
     * and slot_w2 + i*(d*f) elements.  Slots [0, n_cache) are the cache,
     * slots [n_cache, n_cache + n_stage) the staging ring. */
    void* slot_w13;
    void* slot_w2;
    const void* sh_w13;            /* [n_shared][2f][d] device, NULL iff n_shared == 0 */
    const void* sh_w2;             /* [n_shared][d][f] device */
    int32_t layout;                /* caee_layout_t of all of the above */
    int32_t n_cache;               /* >= 0 */
    int32_t n_stage;               /* >= 0; n_cache + n_stage >= 1 */
    int32_t fetch_batch;           /* misses per FFN pass, >= 1 (capped at n_stage when staging is used) */
    float miss_cost;               /* cost-table entry of a non-resident expert, finite and > 0
                                      (e.g. alpha * S_e / B + beta, Sec. IV-A calibration) */
} caee_offload_desc_t;

/* Counters since creation or the last caee_offload_reset. */
typedef struct caee_offload_stats {
    int64_t calls;       /* caee_offload_layer calls with T > 0 */
    int64_t needed;      /* routed experts of A_trans, summed over calls */
    int64_t hits;        /* of them resident when the call began */
    int64_t misses;      /* of them copied host -> device */
    int64_t staged;      /* of the misses, copied into staging slots (not cached) */
    int64_t evictions;   /* cached experts replaced by misses */
    int64_t bytes_h2d;   /* expert bytes copied host -> device */
    int32_t passes;      /* FFN passes of the last call (hits, then one per fetch batch) */
    int32_t reserved;
} caee_offload_stats_t;

/* Creates a handle for layers of shape `desc` (T is ignored here; w_dtype
 * CAEE_F32 or CAEE_BF16).  The cache starts empty.  Host pointers must be
 * page-locked: INVALID_ARG otherwise.  Uses the current device. */
caee_status_t caee_offload_create(const caee_layer_desc_t* desc, const caee_offload_desc_t* od,
                                  caee_offload_t** handle);
/* Waits for the handle's copies and frees what it allocated; NULL is a no-op. */
void caee_offload_destroy(caee_offload_t* handle);
/* One layer call (steps 1-5 above).  desc must match the creating one except
 * for T, tau and importance, and must have n_bins == 1.  `out` may be NULL.
 * `stream` and `copy_stream` must be different streams of the handle's
 * device.  Returns CAEE_ERR_CAPACITY, with the routing outputs written, y
 * not written and the residency unchanged, when the call needs more misses
 * than the free cache slots can take and n_stage is 0.  Blocks the host
 * until the routing step has run. */
caee_status_t caee_offload_layer(caee_offload_t* handle, const caee_layer_desc_t* desc, const void* x,
                                 const float* logits, const float* bias, void* y, const caee_route_out_t* out,
                                 void* ws, size_t ws_bytes, void* stream, void* copy_stream);
caee_status_t caee_offload_stats(const caee_offload_t* handle, caee_offload_stats_t* stats);
/* slot_of [E] host: cache slot holding expert e, or -1. */
caee_status_t caee_offload_residency(const caee_offload_t* handle, int32_t* slot_of);
/* Empties the cache and zeroes the counters (waits for pending copies). */
caee_status_t caee_offload_reset(caee_offload_t* handle);

/* The residency plan of one call, on host arrays (what caee_offload_layer
 * runs in step 3; exposed so it can be checked without a device).
 *   slot_of [E]: in/out, cache slot of each expert or -1;
 *   slot_expert [n_cache], slot_used [n_cache]: in/out, expert held by each
 *     cache slot (-1 empty) and the call index that last needed it;
 *   call: index of this call (larger than every slot_used entry);
 *   need [E]: nonzero for the routed experts of A_trans.
 * Outputs: fetch [E] the misses in copy order (cached ones first, then
 *   staged, each part in ascending expert order), fetch_slot [E] their slot
 *   (staged misses cycle through n_cache .. n_cache+n_stage-1), and counts[4]
 *   = hits, misses, staged, evictions.  Victims are taken in order of
 *   (slot_used, expert) ascending among slots whose expert is not needed;
 *   empty slots, lowest first, before any victim.  CAEE_ERR_CAPACITY (and
 *   nothing changed) if misses exceed the free cache slots and n_stage == 0. */
caee_status_t caee_lru_step(int32_t E, int32_t n_cache, int32_t n_stage, int32_t* slot_of, int32_t* slot_expert,
                            int64_t* slot_used, int64_t call, const uint8_t* need, int32_t* fetch,
                            int32_t* fetch_slot, int32_t* counts);

/* Static description of a status code. */
const char* caee_status_str(caee_status_t status);
/* Message of the last error raised on the calling thread ("" if none). */
const char* caee_last_error(void);
/* CAEE_ABI_VERSION of the built library. */
int caee_abi_version(void);

/* Opt-in per-kernel timing.  While enabled, every kernel the library
 * launches is bracketed by HIP events recorded on the caller's stream.
 * caee_timing_query waits for the recorded events and returns, for kernel
 * kind `kind`, the summed duration in milliseconds and the number of
 * launches since the last reset.  Process-wide state, not thread-safe. */
typedef enum caee_kernel_kind {
    CAEE_KERNEL_ROUTE = 0,    /* routing + pruning + compensation + permutation */
    CAEE_KERNEL_GATE_UP = 1,  /* expert gate/up products and SwiGLU */
    CAEE_KERNEL_DOWN = 2,     /* expert down products */
    CAEE_KERNEL_COMBINE = 3,  /* weighted combine into y */
    CAEE_KERNEL_QUANT = 4,    /* fp8 activation quantisation (x and the SwiGLU rows) */
    CAEE_KERNEL_KINDS = 5
} caee_kernel_kind_t;
caee_status_t caee_timing_enable(int on);
caee_status_t caee_timing_reset(void);
caee_status_t caee_timing_query(int kind, double* total_ms, int64_t* launches);

#ifdef __cplusplus
}
#endif

#endif /* CAEE_H */
