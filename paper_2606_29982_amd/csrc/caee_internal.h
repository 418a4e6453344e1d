// Internal definitions shared by the CAEE host library and its gfx950
// kernels: launch parameter blocks, workspace layout and small device
// helpers (wave reductions, bf16 rounding, MFMA fragments).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <vector>

#include "../../include/caee.h"

namespace caee {

constexpr int kWave = 64;
constexpr int kMaxE = 256;
constexpr int kMaxK = 16;
constexpr int kMaxShared = 4;
constexpr int kMaxBins = 256;
constexpr int kMaxT = 65536;        // tokens per call
constexpr int kMaskT = 1024;        // token block of the permutation (one LDS bitmask per expert)
constexpr int kRouteThreads = 1024;
constexpr int kStats = 9;          // entries of caee_route_out_t.stats
// 16-token MFMA column blocks one FFN work item can hold (1, 2, 4 or 8).
#ifndef CAEE_MAX_TOKEN_BLOCKS
#define CAEE_MAX_TOKEN_BLOCKS 8
#endif
constexpr int kMaxTokenBlocks = CAEE_MAX_TOKEN_BLOCKS;
// Batches above this many tokens use 128-row big chunks (fewer weight
// re-reads, one wave per SIMD); others 64-row chunks (two waves per SIMD),
// which measured faster up to the 4096-token prefill.
#ifndef CAEE_PREFILL_T
#define CAEE_PREFILL_T 65536
#endif
constexpr int kPrefillT = CAEE_PREFILL_T;
// 8-bit batches above this many tokens run their big chunks (as wide as its
// token tile: 256 rows) with the prefill kernel of ffn_prefill8.hip, when the
// weights are tiled and the sizes fit (0 disables it).
#ifndef CAEE_GEMM_T
#define CAEE_GEMM_T 256
#endif
constexpr int kGemmT = CAEE_GEMM_T;
// bf16 big chunks (experts with more rows than a small chunk holds) run
// the same LDS-pipelined GEMM, as wide as its token tile (0 disables).
#ifndef CAEE_GEMM_BF16
#define CAEE_GEMM_BF16 1
#endif
constexpr int kGemmBf16 = CAEE_GEMM_BF16;
// FFN kernel launch (one place to change how the FFN kernels are enqueued).
template <typename K, typename... Args>
inline void ffn_launch(K kernel, dim3 grid, dim3 block, hipStream_t s, Args... args) {
    hipLaunchKernelGGL(kernel, grid, block, 0, s, args...);
}
constexpr int kFfnThreads = 256;    // 4 independent waves per FFN workgroup
#ifndef CAEE_ROUTE_SHARED
#define CAEE_ROUTE_SHARED 1   // batches of up to 16 tokens run the shared experts' gate/up in the routing launch
#endif
constexpr bool kRouteShared = CAEE_ROUTE_SHARED != 0;
// Contraction steps loaded ahead by those workgroups (1024 threads: at most
// 128 registers per lane; 4 spills).
#ifndef CAEE_ROUTE_SHARED_U
#define CAEE_ROUTE_SHARED_U 2
#endif
constexpr int kRouteSharedU = CAEE_ROUTE_SHARED_U;

// Gate/up wave work items wanted per call before the contraction is split
// (about 64 per SIMD: short items keep the tail of the launch short; 64
// measured faster than 32 and 16 at 32 tokens, equal elsewhere).
#ifndef CAEE_TARGET_ITEMS
#define CAEE_TARGET_ITEMS 65536
#endif
constexpr long long kTargetItems = CAEE_TARGET_ITEMS;

// Contraction steps (one 16-byte load per lane) issued together per wave.
#ifndef CAEE_GATE_UP_U
#define CAEE_GATE_UP_U 4
#endif
#ifndef CAEE_DOWN_U
#define CAEE_DOWN_U 8   // 8 loads in flight per lane measured 2 % faster at 32 tokens than 4; 16 slower
#endif
// The same for the decode kernels (one token block), whose contraction
// double-buffers both operands.
#ifndef CAEE_GATE_UP_U1
#define CAEE_GATE_UP_U1 4
#endif
#ifndef CAEE_DOWN_U1
#define CAEE_DOWN_U1 8
#endif
constexpr int kGateUpU = CAEE_GATE_UP_U;
constexpr int kDownU = CAEE_DOWN_U;
#ifndef CAEE_DOWN_AHEAD_NB
#define CAEE_DOWN_AHEAD_NB 1   // down kernels up to this many token blocks double-buffer the H rows too
#endif
constexpr int kGateUpU1 = CAEE_GATE_UP_U1;
constexpr int kDownU1 = CAEE_DOWN_U1;
// Whether the LDS-staged kernels run the big chunks (0: the direct kernels).
#ifndef CAEE_BIG_STAGED
#define CAEE_BIG_STAGED 1
#endif
constexpr bool kBigStaged = CAEE_BIG_STAGED != 0;
// Run the big-chunk launches on a second stream, concurrently with the small ones.
#ifndef CAEE_BIG_CONCURRENT
#define CAEE_BIG_CONCURRENT 1
#endif
constexpr bool kBigConcurrent = CAEE_BIG_CONCURRENT != 0;
constexpr int kFp8U = 2;            // 128-wide fp8 MFMA blocks per step (4 x 16-byte loads per matrix)
// Minimum resident waves per SIMD the FFN kernels are compiled for (0: no bound).
#ifndef CAEE_FFN_WAVES_PER_EU
#define CAEE_FFN_WAVES_PER_EU 0
#endif

// ---------------------------------------------------------------------------
// Workspace layout.  Every region is 256-byte aligned.
struct WsLayout {
    size_t ids, w;              // [T][k] K_final and weights when the caller gives none
    size_t orig;                // [T][k] K_t when the caller gives none
    size_t gbuf;                // [T][k] float64 normalised gate weights G(t)
    size_t top1;                // [T] each token's top expert
    size_t trans;               // [E] uint8 membership of A_trans
    size_t mflag;               // [T][k] uint8: the (token, slot) pair is mandatory on its own
    size_t imp_sum;             // [E] float64 batch-summed gate weight (SUM rule)
    size_t counters;            // [4] int: (unused), refilled slots, empty slots
    size_t perm_off;            // [E + n_shared + 1] first permuted row of each expert slot
    size_t perm_tok;            // [P] token of each permuted row
    size_t perm_pos;            // [T][k + n_shared] permuted row of each (token, slot), -1 unused
    size_t perm_blk;            // [ceil(T / kMaskT)][E] per token block: expert counts, then first rows
    size_t chunks;              // [max_chunks][4] (expert slot, first row, rows, pair): small chunks, then big
    size_t n_chunks;            // [2] small and big chunk counts
    size_t h;                   // [P][f] SwiGLU activations (weight dtype; fp32 for fp8)
    size_t y;                   // [P][d] expert outputs (fp32; bf16 on the 8-bit path)
    size_t xq, xs;              // fp8 path: [T][d] e4m3 codes of x and [T][d/128] fp32 scales
    size_t hq, hs;              // fp8 path: [P][f] e4m3 codes of H and [P][f/128] fp32 scales
    size_t xst, hst;            // fp8 GEMM: [d/128][P] and [f/128][P] block scales of the permuted rows
    size_t total;
    int P, max_chunks, ksplit;
    int chunk_small;            // an expert slot with at most this many rows is one small chunk
    int chunk_big;              // rows of a big chunk at most
};

inline size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

// Bytes per element of the expert output rows Y: bf16 on the 8-bit path,
// where they are the largest intermediate at prefill sizes, else fp32.
inline int y_row_bytes(const caee_layer_desc_t& d) { return d.w_dtype == CAEE_FP8_E4M3 ? 2 : 4; }

// bf16 bits of v, rounded to nearest even (finite values).
__host__ __device__ inline uint32_t bf16_rne(float v) {
    union { float f; uint32_t u; } c;
    c.f = v;
    return (c.u + 0x7FFFu + ((c.u >> 16) & 1u)) >> 16;
}

inline int elem_bytes(int dtype) {
    return dtype == CAEE_F32 ? 4 : dtype == CAEE_BF16 ? 2 : 1;
}

#ifndef CAEE_SPLIT_MAX
#define CAEE_SPLIT_MAX 4   // largest contraction split (the 4 waves of a workgroup); 2 and 1 measured slower at T <= 32
#endif
// Split of the gate/up contraction: when a call has few chunks, the d
// dimension is cut into up to 4 ranges (the waves of one workgroup) so that
// every SIMD gets several work items.  The host fixes the largest split the
// row length allows; the kernels take the split for the number of chunks the
// call actually has (gate_up_split_for), which routing decides on the device.
inline int gate_up_split(const caee_layer_desc_t& d) {
    // Contraction steps of one work item: 64-byte row pieces (one MFMA for
    // bf16) or 128-wide scale blocks (one MFMA for fp8).
    const bool fp8 = d.w_dtype == CAEE_FP8_E4M3;
    const int ksteps = fp8 ? d.d / 128 : d.d * elem_bytes(d.w_dtype) / 64;
    const int U = fp8 ? kFp8U : kGateUpU;
    int S = 1;
    while (S < CAEE_SPLIT_MAX && ksteps % (2 * S * U) == 0) S *= 2;
    return S;
}

__host__ __device__ inline int gate_up_split_for(int n_chunks, int tiles, int s_max) {
    int S = s_max;
    while (S > 1 && (long long)n_chunks * tiles * (S / 2) >= kTargetItems) S >>= 1;
    return S;
}

// Work list of the FFN kernels.  An expert slot with at most
// 16 * small_token_blocks rows of the call is one "small" chunk; a slot with
// more rows is cut into ceil(rows / chunk_big) near-equal "big" chunks of at
// most chunk_big = 16 * big_token_blocks rows.  The two kinds run in
// separate launches, each compiled for its own token-block count: most
// experts of a decode batch carry a handful of tokens, and compiling their
// work items for the hot experts' rows would cost them occupancy.  Each
// chunk streams its expert's weights once.

// 16-token column blocks of the small-chunk kernels (1 or 2).
inline int small_token_blocks(const caee_layer_desc_t& d) { return d.T <= 16 ? 1 : 2; }

// 16-token column blocks of the big-chunk kernels (0: the call has no big
// chunks since no slot can have more rows than T).
inline int big_token_blocks(const caee_layer_desc_t& d) {
    if (d.T <= 16 * small_token_blocks(d)) return 0;
    int nb = d.T <= kPrefillT ? 4 : 8;
    if (kGemmT > 0 && d.w_dtype == CAEE_FP8_E4M3 && d.T > kGemmT) nb = 8;
    return nb < kMaxTokenBlocks ? nb : kMaxTokenBlocks;
}

bool gemm_fp8_applies(const caee_layer_desc_t& d, bool tiled);
bool gemm_bf16_applies(const caee_layer_desc_t& d, bool tiled);
int gemm_fp8_blocks();         // 16-token blocks of an 8-bit big chunk
int gemm_bf16_blocks();        // 16-token blocks of a bf16 big chunk
bool gemm_fp8_fuses_quant();   // the GEMM's gate/up writes the e4m3 H rows itself

// 16-token column blocks of a call's big chunks: the width of the 8-bit
// GEMM's tile when that kernel runs the call's big list (its chunks are as
// wide as its tile), big_token_blocks otherwise.  The chunk lists and the FFN
// launches both take it from here; the workspace is sized for
// big_token_blocks, which never gives fewer chunks.
inline int call_big_blocks(const caee_layer_desc_t& d, bool tiled) {
    const int nb = big_token_blocks(d);
    if (nb > 0 && gemm_fp8_applies(d, tiled)) return gemm_fp8_blocks();
    if (nb > 0 && gemm_bf16_applies(d, tiled)) return gemm_bf16_blocks();
    return nb;
}

// Rows per big chunk of a call (16 when there are no big chunks).
inline int call_chunk_big(const caee_layer_desc_t& d, bool tiled) {
    const int nb = call_big_blocks(d, tiled);
    return 16 * (nb > 0 ? nb : 1);
}

inline WsLayout ws_layout(const caee_layer_desc_t& d) {
    WsLayout L{};
    const size_t T = d.T > 0 ? d.T : 0;
    const int slots = d.k + d.n_shared;
    L.P = int(T * slots);
    L.chunk_small = 16 * small_token_blocks(d);
    L.chunk_big = 16 * (big_token_blocks(d) > 0 ? big_token_blocks(d) : 1);
    // Every expert slot gives one small chunk or ceil(rows / chunk_big) big
    // ones, so the count is at most (slots) + P / chunk_big.
    L.max_chunks = d.E + d.n_shared + (L.P + L.chunk_big - 1) / L.chunk_big;
    size_t off = 0;
    auto take = [&](size_t bytes) { size_t o = off; off += align256(bytes); return o; };
    L.ids = take(T * d.k * 4);
    L.w = take(T * d.k * 4);
    L.orig = take(T * d.k * 4);
    L.gbuf = take(T * d.k * 8);
    L.top1 = take(T * 4);
    L.trans = take(d.E);
    L.mflag = take(T * d.k);
    L.imp_sum = take(size_t(d.E) * 8);
    L.counters = take(16);
    L.perm_off = take(size_t(d.E + d.n_shared + 1) * 4);
    L.perm_tok = take(size_t(L.P) * 4);
    L.perm_pos = take(T * slots * 4);
    L.perm_blk = take(((T + kMaskT - 1) / kMaskT) * size_t(d.E) * 4);
    L.chunks = take(size_t(L.max_chunks) * 16);
    L.n_chunks = take(16);
    const int h_bytes = d.w_dtype == CAEE_FP8_E4M3 ? 4 : elem_bytes(d.w_dtype);
    L.h = take(size_t(L.P) * d.f * h_bytes);
    L.y = take(size_t(L.P) * d.d * y_row_bytes(d));
    const bool fp8 = d.w_dtype == CAEE_FP8_E4M3;
    L.xq = take(fp8 ? T * d.d : 0);
    L.xs = take(fp8 ? T * (d.d / 128) * 4 : 0);
    L.hq = take(fp8 ? size_t(L.P) * d.f : 0);
    L.hs = take(fp8 ? size_t(L.P) * (d.f / 128) * 4 : 0);
    const bool gemm = fp8 && kGemmT > 0 && d.T > kGemmT;
    L.xst = take(gemm ? size_t(L.P) * (d.d / 128) * 4 : 0);
    L.hst = take(gemm ? size_t(L.P) * (d.f / 128) * 4 : 0);
    L.ksplit = gate_up_split(d);
    L.total = off;
    return L;
}

// ---------------------------------------------------------------------------
// Launch parameter blocks (passed by value).
struct RouteParams {
    int T, E, n_group, topk_group, k, n_shared, n_bins;
    int epl;        // experts held per lane (1, 2 or 4)
    int lpg;        // lanes per group (power of two)
    int gsize;      // experts per group
    double rs, tau;
    int rule;       // caee_importance_t
    int refill;     // caee_refill_t
    uint32_t seed;  // random refill keys
    int keep_top1;  // each token's top expert mandatory in every call (else only when A_trans comes out empty)
    const float* logits;
    const float* bias;
    const float* cost;
    const int32_t* bin;
    // routing outputs
    int32_t* topk_ids;
    float* topk_w;
    int32_t* orig_ids;
    uint32_t* masks;
    int32_t* stats;
    double* bin_loads;
    // per-call scratch
    double* gbuf;
    int32_t* top1;
    uint8_t* trans;
    uint8_t* mflag;
    double* imp_sum;
    int32_t* counters;
    int chunk_small, chunk_big;
    // permutation outputs
    int32_t* perm_off;
    int32_t* perm_tok;
    int32_t* perm_pos;
    int32_t* perm_blk;
    int32_t* chunks;
    int32_t* n_chunks;
    double* sslot;      // scores s of each token's K_t slots [T][k] when kept by routing (else recomputed)
    int do_permute;     // 0: the permutation kernel only reports the refill/empty-slot counts
};

struct FfnParams {
    int T, d, f, E, k, n_shared;
    const void* x;
    const void* w13;
    const void* w2;
    const void* sh_w13;
    const void* sh_w2;
    const float* w13_scale;
    const float* w2_scale;
    const float* sh_w13_scale;
    const float* sh_w2_scale;
    const int32_t* perm_tok;
    const int32_t* perm_pos;
    const int32_t* chunks;
    const int32_t* n_chunks;
    int list;         // 0: the small chunks, 1: the big chunks
    const int32_t* topk_ids;
    const float* topk_w;
    void* h;
    void* yperm;      // [P][d] expert output rows, fp32 (bf16 when y_half)
    void* y;
    int y_bf16;
    int P;
    int ksplit;
    int tiled;      // weights in CAEE_LAYOUT_TILED order
    // Offload residency: when wtab is set, expert slot x takes its w13 / w2
    // base from wtab[2x] / wtab[2x+1] instead of the contiguous arrays, and
    // when pass_of is set only chunks of slots with pass_of[x] == pass_id run.
    const void* const* wtab;
    const int32_t* pass_of;
    int pass_id;
    // fp8 path: quantised activations and their per-token 128-channel scales
    uint8_t* xq;
    float* xs;
    uint8_t* hq;
    float* hs;
    float* xst;       // 8-bit GEMM: block scales transposed, [block][permuted row]
    float* hst;
    int skip_shared;  // chunks of shared slots are skipped (their gate/up already ran)
    int y_half;       // the expert output rows are bf16 (8-bit path): half the traffic of the combine
};

// ---------------------------------------------------------------------------
// FFN work items: chunk c of the list a launch runs (the small chunks are
// listed first, then the big ones).
struct ChunkRef {
    int xs, row0, ntok;
    int pair;   // list offset (+1 / -1) of the other piece of a pair, 0 if unpaired
};

__device__ inline int ffn_list_size(const FfnParams& p) { return p.n_chunks[p.list]; }

__device__ inline ChunkRef ffn_chunk(const FfnParams& p, int c) {
    const int32_t* ch = p.chunks + 4 * ((p.list ? p.n_chunks[0] : 0) + c);
    return {ch[0], ch[1], ch[2], ch[3]};
}

// Token of permuted row `row` (of expert slot xs).
__device__ inline int ffn_token(const FfnParams& p, int xs, int row) {
    (void)xs;
    return p.perm_tok[row];
}

// Offload passes: only the chunks of experts in pass p.pass_id run; with
// skip_shared, no chunk of a shared slot.
__device__ inline bool ffn_skip(const FfnParams& p, int xs) {
    return (p.skip_shared && xs >= p.E) || (p.pass_of && p.pass_of[xs] != p.pass_id);
}

// First byte of matrix w13 (w2 = false) or w2 of expert slot xs.
__device__ inline const char* ffn_weights(const FfnParams& p, int xs, bool w2, size_t expert_bytes) {
    if (xs >= p.E) return (const char*)(w2 ? p.sh_w2 : p.sh_w13) + (size_t)(xs - p.E) * expert_bytes;
    if (p.wtab) return (const char*)p.wtab[2 * xs + (w2 ? 1 : 0)];
    return (const char*)(w2 ? p.w2 : p.w13) + (size_t)xs * expert_bytes;
}

// Four consecutive outputs of expert output row `row`, column `col`.
__device__ inline void store_y4(const FfnParams& p, size_t row, int col, float a, float b, float c, float e) {
    const size_t o = row * p.d + col;
    if (p.y_half) {
        uint2 pk;
        pk.x = bf16_rne(a) | (bf16_rne(b) << 16);
        pk.y = bf16_rne(c) | (bf16_rne(e) << 16);
        *(uint2*)((uint16_t*)p.yperm + o) = pk;
    } else {
        *(float4*)((float*)p.yperm + o) = make_float4(a, b, c, e);
    }
}

__device__ inline float4 load_y4(const FfnParams& p, size_t row, int col) {
    const size_t o = row * p.d + col;
    if (p.y_half) {
        const uint2 pk = *(const uint2*)((const uint16_t*)p.yperm + o);
        return make_float4(__uint_as_float(pk.x << 16), __uint_as_float(pk.x & 0xFFFF0000u),
                           __uint_as_float(pk.y << 16), __uint_as_float(pk.y & 0xFFFF0000u));
    }
    return *(const float4*)((const float*)p.yperm + o);
}

__device__ inline const float* ffn_scales(const FfnParams& p, int xs, bool w2, size_t per_expert) {
    if (xs >= p.E) return (w2 ? p.sh_w2_scale : p.sh_w13_scale) + (size_t)(xs - p.E) * per_expert;
    return (w2 ? p.w2_scale : p.w13_scale) + (size_t)xs * per_expert;
}

// Host-side launchers (defined next to their kernels).
hipError_t launch_route(const RouteParams& p, hipStream_t s);
// Small batches: the single-workgroup routing launch also runs the shared
// experts' gate/up (their rows hold every token and come first, so they
// need nothing routing computes) in workgroups of its own.
bool route_runs_shared(const caee_layer_desc_t& d);
hipError_t launch_route_shared(const RouteParams& p, const FfnParams& fp, int w_dtype, hipStream_t s);
hipError_t launch_permute(const RouteParams& p, hipStream_t s);
hipError_t launch_gate_up(const FfnParams& p, int w_dtype, int nb, int max_chunks, hipStream_t s);
hipError_t launch_down(const FfnParams& p, int w_dtype, int nb, int max_chunks, hipStream_t s);
hipError_t launch_combine(const FfnParams& p, hipStream_t s);
hipError_t launch_quant_rows(const void* src, int src_bf16, long long rows, int cols, uint8_t* q, float* scale,
                             hipStream_t s);
hipError_t launch_gate_up_fp8(const FfnParams& p, int nb, int max_chunks, hipStream_t s);
hipError_t launch_quant_list(const FfnParams& p, int nb, int max_chunks, bool transposed, hipStream_t s);
hipError_t launch_gather_xs(const FfnParams& p, int max_chunks, hipStream_t s);
bool gemm_fp8_supports(const FfnParams& p, int nb);
bool gemm_bf16_supports(const FfnParams& p, int nb);
hipError_t launch_gemm(const FfnParams& p, bool gate_up, int max_chunks, hipStream_t s);   // bf16 big chunks
hipError_t launch_prefill8(const FfnParams& p, bool gate_up, int max_chunks, hipStream_t s);
hipError_t launch_down_fp8(const FfnParams& p, int nb, int max_chunks, hipStream_t s);
hipError_t launch_pack(const void* src, void* dst, long long rows, long long row_units, long long count,
                       hipStream_t s);
int device_cu_count();

// ---------------------------------------------------------------------------
// Host helpers shared by the entry points (defined in api.hip).
caee_status_t fail(caee_status_t st, const char* fmt, ...);
caee_status_t check_desc(const caee_layer_desc_t* d);
caee_status_t check_ptr(const void* p, const char* name, bool required);
caee_status_t check_ws(const caee_layer_desc_t* d, void* ws, size_t ws_bytes, WsLayout* L);
caee_status_t check_route_inputs(const caee_layer_desc_t* d, const float* logits, const float* bias,
                                 const float* cost, const int32_t* bin);
caee_status_t check_route_out(const caee_route_out_t* out);
void clear_last_error();
RouteParams make_route_params(const caee_layer_desc_t* d, const float* logits, const float* bias,
                              const float* cost, const int32_t* bin, char* ws, const WsLayout& L);
FfnParams make_ffn_params(const caee_layer_desc_t* d, const void* x, const int32_t* ids, const float* w,
                          const caee_expert_weights_t* W, void* y, char* ws, const WsLayout& L);
// Routing, pruning, compensation and permutation of a whole-layer call; the
// routing results go to `out` when given, else to the workspace.
caee_status_t run_route_layer(const caee_layer_desc_t* d, RouteParams& p, const caee_route_out_t* out, char* ws,
                              const WsLayout& L, hipStream_t s, const FfnParams* shared_fp = nullptr);
void set_route_outputs(RouteParams& p, const caee_route_out_t* out, char* ws, const WsLayout& L);

// The FFN of one layer call, in three parts:
//   ffn_begin   (fp8) quantises x;
//   ffn_routed  after the permutation, runs the small chunks on the main
//               stream and (big_on_side) the big chunks on a side stream
//               forked from it; with p.pass_of set only pass p.pass_id runs;
//   ffn_end     joins the side stream and combines into y.
struct FfnCall {
    hipStream_t main = nullptr, side = nullptr;   // side == main until forked
    hipEvent_t ev_join = nullptr;
    bool shared_done = false;   // the routing launch already ran the shared experts' gate/up
};
caee_status_t ffn_begin(const caee_layer_desc_t* d, const FfnParams& p, const WsLayout& L, hipStream_t s,
                        FfnCall* call);
caee_status_t ffn_routed(const caee_layer_desc_t* d, const FfnParams& p, const WsLayout& L, FfnCall* call,
                         bool big_on_side);
caee_status_t ffn_end(const FfnParams& p, FfnCall* call);

// Opt-in timing: events bracket each launch on the caller's stream.
struct TimingRec {
    int kind;
    hipEvent_t a, b;
};
struct Timing {
    bool on = false;
    std::vector<TimingRec> pending;
    std::vector<hipEvent_t> pool;
    double total_ms[CAEE_KERNEL_KINDS] = {};
    int64_t launches[CAEE_KERNEL_KINDS] = {};
};
Timing& timing();
hipEvent_t take_event();
bool timing_suppressed();   // the calling thread runs a call that must create no events

// Runs one launch, bracketed by timing events when timing is on.
template <class F>
caee_status_t timed_launch(int kind, hipStream_t s, const char* what, F&& launch) {
    Timing& tm = timing();
    hipEvent_t a = nullptr, b = nullptr;
    bool timed = false;
    if (tm.on && !timing_suppressed()) {
        a = take_event();
        b = take_event();
        timed = a && b && hipEventRecord(a, s) == hipSuccess;
    }
    const hipError_t err = launch();
    if (err != hipSuccess) return fail(CAEE_ERR_HIP, "%s launch failed: %s", what, hipGetErrorString(err));
    if (timed && hipEventRecord(b, s) == hipSuccess) {
        tm.pending.push_back({kind, a, b});
    } else {
        if (a) tm.pool.push_back(a);
        if (b) tm.pool.push_back(b);
    }
    return CAEE_OK;
}

#define CAEE_TRY(expr)                          \
    do {                                        \
        caee_status_t st_ = (expr);             \
        if (st_ != CAEE_OK) return st_;         \
    } while (0)

}  // namespace caee
