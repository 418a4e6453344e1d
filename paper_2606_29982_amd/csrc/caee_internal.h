// Internal definitions shared by the CAEE host library and its gfx950
// kernels: launch parameter blocks, workspace layout and small device
// helpers (wave reductions, bf16 rounding, MFMA fragments).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/caee.h"

namespace caee {

constexpr int kWave = 64;
constexpr int kMaxE = 256;
constexpr int kMaxK = 16;
constexpr int kMaxShared = 4;
constexpr int kMaxBins = 256;
constexpr int kFusedMaxT = 128;     // routing + permutation in one workgroup
constexpr int kRouteThreads = 1024;
constexpr int kChunkTokens = 128;   // tokens of one expert handled by one FFN work item
constexpr int kFfnThreads = 256;    // 4 independent waves per FFN workgroup

// ---------------------------------------------------------------------------
// Workspace layout.  Every region is 256-byte aligned.
struct WsLayout {
    size_t ids, w;              // [T][k] K_final and weights when the caller gives none
    size_t orig;                // [T][k] K_t when the caller gives none
    size_t perm_off;            // [E + n_shared + 1] first permuted row of each expert slot
    size_t perm_tok;            // [P] token of each permuted row
    size_t perm_pos;            // [T][k + n_shared] permuted row of each (token, slot), -1 unused
    size_t chunks;              // [max_chunks][4] (expert slot, first row, rows, 0)
    size_t n_chunks;            // [1]
    size_t h;                   // [P][f] SwiGLU activations (weight dtype; fp32 for fp8)
    size_t y;                   // [P][d] fp32 expert outputs
    size_t total;
    int P, max_chunks;
};

inline size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

inline int elem_bytes(int dtype) {
    return dtype == CAEE_F32 ? 4 : dtype == CAEE_BF16 ? 2 : 1;
}

inline WsLayout ws_layout(const caee_layer_desc_t& d) {
    WsLayout L{};
    const size_t T = d.T > 0 ? d.T : 0;
    const int slots = d.k + d.n_shared;
    L.P = int(T * slots);
    L.max_chunks = d.E + d.n_shared + (L.P + kChunkTokens - 1) / kChunkTokens;
    size_t off = 0;
    auto take = [&](size_t bytes) { size_t o = off; off += align256(bytes); return o; };
    L.ids = take(T * d.k * 4);
    L.w = take(T * d.k * 4);
    L.orig = take(T * d.k * 4);
    L.perm_off = take(size_t(d.E + d.n_shared + 1) * 4);
    L.perm_tok = take(size_t(L.P) * 4);
    L.perm_pos = take(T * slots * 4);
    L.chunks = take(size_t(L.max_chunks) * 16);
    L.n_chunks = take(16);
    const int h_bytes = d.w_dtype == CAEE_FP8_E4M3 ? 4 : elem_bytes(d.w_dtype);
    L.h = take(size_t(L.P) * d.f * h_bytes);
    L.y = take(size_t(L.P) * d.d * 4);
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
    // permutation outputs
    int32_t* perm_off;
    int32_t* perm_tok;
    int32_t* perm_pos;
    int32_t* chunks;
    int32_t* n_chunks;
    int do_route;       // 0: read K_final from topk_ids instead of routing
    int do_permute;
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
    const int32_t* topk_ids;
    const float* topk_w;
    void* h;
    float* yperm;
    void* y;
    int y_bf16;
};

// Host-side launchers (defined next to their kernels).
hipError_t launch_route(const RouteParams& p, hipStream_t s);
hipError_t launch_gate_up(const FfnParams& p, int w_dtype, int max_chunks, hipStream_t s);
hipError_t launch_down(const FfnParams& p, int w_dtype, int max_chunks, hipStream_t s);
hipError_t launch_combine(const FfnParams& p, hipStream_t s);
int device_cu_count();

}  // namespace caee
