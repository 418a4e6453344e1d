// Host side of the CAEE C ABI: argument validation, workspace carving,
// launch order and opt-in per-kernel timing.  No device memory is allocated
// here; every buffer is the caller's.
#include <math.h>

#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <string>
#include <vector>

#include "caee_internal.h"

namespace caee {


namespace {
thread_local std::string g_last_error;
// Set while the no-allocation entry point runs: opt-in timing (which
// creates HIP events) stays off for its launches.
thread_local bool g_no_timing = false;

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

int experts_per_lane(int E) { return E <= 64 ? 1 : E <= 128 ? 2 : 4; }
}  // namespace

void clear_last_error() { g_last_error.clear(); }

caee_status_t fail(caee_status_t st, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return st;
}

caee_status_t check_desc(const caee_layer_desc_t* d) {
    if (!d) return fail(CAEE_ERR_INVALID_ARG, "desc is NULL");
    if (d->T < 0) return fail(CAEE_ERR_INVALID_ARG, "T=%d must be >= 0", d->T);
    if (d->d <= 0 || d->d % 128) return fail(CAEE_ERR_INVALID_ARG, "d=%d must be a positive multiple of 128", d->d);
    if (d->f <= 0 || d->f % 128) return fail(CAEE_ERR_INVALID_ARG, "f=%d must be a positive multiple of 128", d->f);
    if (d->E < 1 || d->E > kMaxE) return fail(CAEE_ERR_INVALID_ARG, "E=%d must be in [1, %d]", d->E, kMaxE);
    if (d->n_group < 1 || d->E % d->n_group)
        return fail(CAEE_ERR_INVALID_ARG, "n_group=%d must divide E=%d", d->n_group, d->E);
    if (d->topk_group < 1 || d->topk_group > d->n_group)
        return fail(CAEE_ERR_INVALID_ARG, "topk_group=%d must be in [1, n_group=%d]", d->topk_group, d->n_group);
    const int gsize = d->E / d->n_group;
    if (d->k < 1 || d->k > kMaxK || d->k > d->topk_group * gsize)
        return fail(CAEE_ERR_INVALID_ARG, "k=%d must be in [1, min(%d, topk_group*E/n_group=%d)]", d->k, kMaxK,
                    d->topk_group * gsize);
    if (d->n_shared < 0 || d->n_shared > kMaxShared)
        return fail(CAEE_ERR_INVALID_ARG, "n_shared=%d must be in [0, %d]", d->n_shared, kMaxShared);
    if (!(isfinite(d->routed_scaling) && d->routed_scaling > 0.0f))
        return fail(CAEE_ERR_INVALID_ARG, "routed_scaling must be finite and > 0");
    if (!(isfinite(d->tau) && d->tau >= 0.0f)) return fail(CAEE_ERR_INVALID_ARG, "tau must be finite and >= 0");
    if (d->n_bins < 1 || d->n_bins > kMaxBins)
        return fail(CAEE_ERR_INVALID_ARG, "n_bins=%d must be in [1, %d]", d->n_bins, kMaxBins);
    if (d->importance != CAEE_IMPORTANCE_MAX && d->importance != CAEE_IMPORTANCE_SUM &&
        d->importance != CAEE_IMPORTANCE_CIR)
        return fail(CAEE_ERR_INVALID_ARG, "unknown importance=%d", d->importance);
    if (d->refill != CAEE_REFILL_SCORE && d->refill != CAEE_REFILL_NONE && d->refill != CAEE_REFILL_RANDOM &&
        d->refill != CAEE_REFILL_LITERAL)
        return fail(CAEE_ERR_INVALID_ARG, "unknown refill=%d", d->refill);
    if (d->keep_top1 != 0 && d->keep_top1 != 1)
        return fail(CAEE_ERR_INVALID_ARG, "keep_top1=%d must be 0 or 1", d->keep_top1);
    if (d->w_dtype != CAEE_F32 && d->w_dtype != CAEE_BF16 && d->w_dtype != CAEE_FP8_E4M3)
        return fail(CAEE_ERR_INVALID_ARG, "unknown w_dtype=%d", d->w_dtype);
    const int want_x = d->w_dtype == CAEE_F32 ? CAEE_F32 : CAEE_BF16;
    if (d->x_dtype != want_x)
        return fail(CAEE_ERR_INVALID_ARG, "x_dtype=%d does not match w_dtype=%d (f32 weights take f32 x, "
                    "bf16/fp8 weights take bf16 x)", d->x_dtype, d->w_dtype);
    if (d->y_dtype != CAEE_F32 && d->y_dtype != CAEE_BF16)
        return fail(CAEE_ERR_INVALID_ARG, "y_dtype=%d must be CAEE_F32 or CAEE_BF16", d->y_dtype);
    // Limits of this build.
    const int epl = experts_per_lane(d->E);
    const int lpg = gsize / epl;
    if (d->E % epl || gsize % epl || (lpg & (lpg - 1)))
        return fail(CAEE_ERR_UNSUPPORTED, "E=%d with %d experts per group needs the group size to be a "
                    "multiple of %d with a power-of-two quotient", d->E, gsize, epl);
    if (d->T > kMaxT) return fail(CAEE_ERR_UNSUPPORTED, "T=%d exceeds %d", d->T, kMaxT);
    return CAEE_OK;
}

caee_status_t check_ptr(const void* p, const char* name, bool required) {
    if (!p) return required ? fail(CAEE_ERR_INVALID_ARG, "%s is NULL", name) : CAEE_OK;
    if (!aligned16(p)) return fail(CAEE_ERR_INVALID_ARG, "%s is not 16-byte aligned", name);
    return CAEE_OK;
}

caee_status_t check_ws(const caee_layer_desc_t* d, void* ws, size_t ws_bytes, WsLayout* L) {
    *L = ws_layout(*d);
    if (!ws) return fail(CAEE_ERR_WORKSPACE, "workspace is NULL");
    if (((uintptr_t)ws & 255u) != 0) return fail(CAEE_ERR_WORKSPACE, "workspace is not 256-byte aligned");
    if (ws_bytes < L->total)
        return fail(CAEE_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", ws_bytes, L->total);
    return CAEE_OK;
}

caee_status_t check_route_inputs(const caee_layer_desc_t* d, const float* logits, const float* bias,
                                 const float* cost, const int32_t* bin) {
    CAEE_TRY(check_ptr(logits, "logits", true));
    CAEE_TRY(check_ptr(bias, "bias", false));
    CAEE_TRY(check_ptr(cost, "cost", true));
    CAEE_TRY(check_ptr(bin, "bin", false));
    if (!bin && d->n_bins != 1) return fail(CAEE_ERR_INVALID_ARG, "bin is NULL but n_bins=%d", d->n_bins);
    return CAEE_OK;
}

caee_status_t check_route_out(const caee_route_out_t* out) {
    if (!out) return fail(CAEE_ERR_INVALID_ARG, "out is NULL");
    CAEE_TRY(check_ptr(out->topk_ids, "out->topk_ids", true));
    CAEE_TRY(check_ptr(out->topk_w, "out->topk_w", true));
    CAEE_TRY(check_ptr(out->orig_ids, "out->orig_ids", false));
    CAEE_TRY(check_ptr(out->masks, "out->masks", false));
    CAEE_TRY(check_ptr(out->stats, "out->stats", false));
    CAEE_TRY(check_ptr(out->bin_loads, "out->bin_loads", false));
    return CAEE_OK;
}

caee_status_t check_weights(const caee_layer_desc_t* d, const caee_expert_weights_t* w) {
    if (!w) return fail(CAEE_ERR_INVALID_ARG, "weights is NULL");
    const bool fp8 = d->w_dtype == CAEE_FP8_E4M3;
    const bool sh = d->n_shared > 0;
    CAEE_TRY(check_ptr(w->w13, "weights->w13", true));
    CAEE_TRY(check_ptr(w->w2, "weights->w2", true));
    CAEE_TRY(check_ptr(w->sh_w13, "weights->sh_w13", sh));
    CAEE_TRY(check_ptr(w->sh_w2, "weights->sh_w2", sh));
    if (!sh && (w->sh_w13 || w->sh_w2)) return fail(CAEE_ERR_INVALID_ARG, "shared weights given with n_shared=0");
    CAEE_TRY(check_ptr(w->w13_scale, "weights->w13_scale", fp8));
    CAEE_TRY(check_ptr(w->w2_scale, "weights->w2_scale", fp8));
    CAEE_TRY(check_ptr(w->sh_w13_scale, "weights->sh_w13_scale", fp8 && sh));
    CAEE_TRY(check_ptr(w->sh_w2_scale, "weights->sh_w2_scale", fp8 && sh));
    if (!fp8 && (w->w13_scale || w->w2_scale || w->sh_w13_scale || w->sh_w2_scale))
        return fail(CAEE_ERR_INVALID_ARG, "block scales given for non-fp8 weights");
    if (w->layout != CAEE_LAYOUT_ROWMAJOR && w->layout != CAEE_LAYOUT_TILED)
        return fail(CAEE_ERR_INVALID_ARG, "unknown weight layout=%d", w->layout);
    return CAEE_OK;
}

Timing& timing() {
    static Timing t;
    return t;
}

bool timing_suppressed() { return g_no_timing; }

hipEvent_t take_event() {
    Timing& tm = timing();
    if (!tm.pool.empty()) {
        hipEvent_t e = tm.pool.back();
        tm.pool.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

namespace {
hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }
}  // namespace

RouteParams make_route_params(const caee_layer_desc_t* d, const float* logits, const float* bias,
                              const float* cost, const int32_t* bin, char* ws, const WsLayout& L) {
    RouteParams p{};
    p.T = d->T;
    p.E = d->E;
    p.n_group = d->n_group;
    p.topk_group = d->topk_group;
    p.k = d->k;
    p.n_shared = d->n_shared;
    p.n_bins = d->n_bins;
    p.epl = experts_per_lane(d->E);
    p.gsize = d->E / d->n_group;
    p.lpg = p.gsize / p.epl;
    p.rs = (double)d->routed_scaling;
    p.tau = (double)d->tau;
    p.logits = logits;
    p.bias = bias;
    p.cost = cost;
    p.bin = bin;
    p.perm_off = (int32_t*)(ws + L.perm_off);
    p.perm_tok = (int32_t*)(ws + L.perm_tok);
    p.perm_pos = (int32_t*)(ws + L.perm_pos);
    p.perm_blk = (int32_t*)(ws + L.perm_blk);
    p.chunks = (int32_t*)(ws + L.chunks);
    p.n_chunks = (int32_t*)(ws + L.n_chunks);
    p.gbuf = (double*)(ws + L.gbuf);
    p.top1 = (int32_t*)(ws + L.top1);
    p.trans = (uint8_t*)(ws + L.trans);
    p.mflag = (uint8_t*)(ws + L.mflag);
    p.imp_sum = (double*)(ws + L.imp_sum);
    p.rule = d->importance;
    p.refill = d->refill;
    p.seed = d->seed;
    p.keep_top1 = d->keep_top1;
    p.counters = (int32_t*)(ws + L.counters);
    p.chunk_small = L.chunk_small;
    p.chunk_big = L.chunk_big;
    p.orig_ids = (int32_t*)(ws + L.orig);
    return p;
}

FfnParams make_ffn_params(const caee_layer_desc_t* d, const void* x, const int32_t* ids, const float* w,
                          const caee_expert_weights_t* W, void* y, char* ws, const WsLayout& L) {
    FfnParams p{};
    p.T = d->T;
    p.d = d->d;
    p.f = d->f;
    p.E = d->E;
    p.k = d->k;
    p.n_shared = d->n_shared;
    p.x = x;
    if (W) {
        p.w13 = W->w13;
        p.w2 = W->w2;
        p.sh_w13 = W->sh_w13;
        p.sh_w2 = W->sh_w2;
        p.w13_scale = W->w13_scale;
        p.w2_scale = W->w2_scale;
        p.sh_w13_scale = W->sh_w13_scale;
        p.sh_w2_scale = W->sh_w2_scale;
        p.tiled = W->layout == CAEE_LAYOUT_TILED;
    }
    p.perm_tok = (const int32_t*)(ws + L.perm_tok);
    p.perm_pos = (const int32_t*)(ws + L.perm_pos);
    p.chunks = (const int32_t*)(ws + L.chunks);
    p.n_chunks = (const int32_t*)(ws + L.n_chunks);
    p.topk_ids = ids;
    p.topk_w = w;
    p.h = ws + L.h;
    p.yperm = ws + L.y;
    p.y_half = y_row_bytes(*d) == 2;
    p.y = y;
    p.y_bf16 = d->y_dtype == CAEE_BF16;
    p.P = L.P;
    p.ksplit = L.ksplit;
    p.xq = (uint8_t*)(ws + L.xq);
    p.xs = (float*)(ws + L.xs);
    p.hq = (uint8_t*)(ws + L.hq);
    p.hs = (float*)(ws + L.hs);
    p.xst = (float*)(ws + L.xst);
    p.hst = (float*)(ws + L.hst);
    return p;
}

namespace {
// A second stream per device and host thread, with the events that fork work
// onto it and join it back.  Created on first use,
// kept until the process ends; default priority.
struct SideStream {
    hipStream_t stream = nullptr;
    hipEvent_t fork = nullptr, join = nullptr;
};

caee_status_t side_stream(SideStream** out) {
    thread_local SideStream per_dev[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return fail(CAEE_ERR_HIP, "hipGetDevice failed");
    SideStream& ss = per_dev[dev];
    if (!ss.stream) {
        hipError_t e = hipStreamCreateWithFlags(&ss.stream, hipStreamNonBlocking);
        if (e == hipSuccess) e = hipEventCreateWithFlags(&ss.fork, hipEventDisableTiming);
        if (e == hipSuccess) e = hipEventCreateWithFlags(&ss.join, hipEventDisableTiming);
        if (e != hipSuccess) {
            ss = SideStream{};
            return fail(CAEE_ERR_HIP, "side stream creation failed: %s", hipGetErrorString(e));
        }
    }
    *out = &ss;
    return CAEE_OK;
}

caee_status_t order(hipEvent_t ev, hipStream_t from, hipStream_t to, const char* what) {
    hipError_t e = hipEventRecord(ev, from);
    if (e == hipSuccess) e = hipStreamWaitEvent(to, ev, 0);
    if (e != hipSuccess) return fail(CAEE_ERR_HIP, "%s failed: %s", what, hipGetErrorString(e));
    return CAEE_OK;
}

caee_status_t gate_up_list(const caee_layer_desc_t* d, FfnParams p, int list, int nb, int max_chunks,
                           hipStream_t s) {
    const int kind = CAEE_KERNEL_GATE_UP;
    p.list = list;
    if (d->w_dtype == CAEE_FP8_E4M3)
        return timed_launch(kind, s, "gate/up", [&] { return launch_gate_up_fp8(p, nb, max_chunks, s); });
    return timed_launch(kind, s, "gate/up", [&] { return launch_gate_up(p, d->w_dtype, nb, max_chunks, s); });
}

caee_status_t down_list(const caee_layer_desc_t* d, FfnParams p, int list, int nb, int max_chunks, hipStream_t s) {
    p.list = list;
    if (d->w_dtype == CAEE_FP8_E4M3)
        return timed_launch(CAEE_KERNEL_DOWN, s, "down", [&] { return launch_down_fp8(p, nb, max_chunks, s); });
    return timed_launch(CAEE_KERNEL_DOWN, s, "down", [&] { return launch_down(p, d->w_dtype, nb, max_chunks, s); });
}

}  // namespace

caee_status_t ffn_begin(const caee_layer_desc_t* d, const FfnParams& p, const WsLayout& L, hipStream_t s,
                        FfnCall* call) {
    (void)L;
    *call = FfnCall{};
    call->main = s;
    call->side = s;
    if (d->w_dtype == CAEE_FP8_E4M3)
        CAEE_TRY(timed_launch(CAEE_KERNEL_QUANT, s, "quantise x",
                              [&] { return launch_quant_rows(p.x, 1, d->T, d->d, p.xq, p.xs, s); }));
    return CAEE_OK;
}

caee_status_t ffn_routed(const caee_layer_desc_t* d, const FfnParams& p, const WsLayout& L, FfnCall* call,
                         bool big_on_side) {
    const int nb_small = small_token_blocks(*d), nb_big = call_big_blocks(*d, p.tiled);
    hipStream_t s = call->main;
    // The big chunks (few, long, latency-bound work items) run on a side
    // stream next to the small ones (many, bandwidth-bound): disjoint rows.
    // The fork comes after routing, which built their list.
    hipStream_t sb = s;
    if (nb_big && big_on_side && kBigConcurrent) {
        SideStream* ss = nullptr;
        CAEE_TRY(side_stream(&ss));
        call->side = ss->stream;
        call->ev_join = ss->join;
        CAEE_TRY(order(ss->fork, s, ss->stream, "fork to the side stream"));
        sb = call->side;
    }
    // Gate/up skips the shared experts when the routing launch ran them.
    FfnParams pg = p;
    pg.skip_shared = call->shared_done ? 1 : 0;
    // One list's chain: gate/up, (fp8) quantisation of its SwiGLU rows, down.
    // The 8-bit GEMM reads its rows' block scales transposed and in permuted
    // row order: gathered once for x, written so by the quantiser for H.
    auto chain = [&](int list, int nb, hipStream_t st) -> caee_status_t {
        const bool gemm = d->w_dtype == CAEE_FP8_E4M3 && nb == gemm_fp8_blocks() && gemm_fp8_applies(*d, p.tiled);
        FfnParams q = p;
        q.list = list;
        if (gemm)
            CAEE_TRY(timed_launch(CAEE_KERNEL_QUANT, st, "gather x scales",
                                  [&] { return launch_gather_xs(q, L.max_chunks, st); }));
        CAEE_TRY(gate_up_list(d, pg, list, nb, L.max_chunks, st));
        if (d->w_dtype == CAEE_FP8_E4M3 && !(gemm && gemm_fp8_fuses_quant()))
            CAEE_TRY(timed_launch(CAEE_KERNEL_QUANT, st, "quantise H",
                                  [&] { return launch_quant_list(q, nb, L.max_chunks, gemm, st); }));
        return down_list(d, p, list, nb, L.max_chunks, st);
    };
    if (nb_big) CAEE_TRY(chain(1, nb_big, sb));
    return chain(0, nb_small, s);
}

caee_status_t ffn_end(const FfnParams& p, FfnCall* call) {
    if (call->side != call->main) CAEE_TRY(order(call->ev_join, call->side, call->main, "join from the side stream"));
    return timed_launch(CAEE_KERNEL_COMBINE, call->main, "combine", [&] { return launch_combine(p, call->main); });
}

void set_route_outputs(RouteParams& p, const caee_route_out_t* out, char* ws, const WsLayout& L) {
    p.topk_ids = out ? out->topk_ids : (int32_t*)(ws + L.ids);
    p.topk_w = out ? out->topk_w : (float*)(ws + L.w);
    if (out && out->orig_ids) p.orig_ids = out->orig_ids;
    p.masks = out ? out->masks : nullptr;
    p.stats = out ? out->stats : nullptr;
    p.bin_loads = out ? out->bin_loads : nullptr;
}

caee_status_t run_route_layer(const caee_layer_desc_t* d, RouteParams& p, const caee_route_out_t* out, char* ws,
                              const WsLayout& L, hipStream_t s, const FfnParams* shared_fp) {
    set_route_outputs(p, out, ws, L);
    p.do_permute = 1;
    if (shared_fp)
        return timed_launch(CAEE_KERNEL_ROUTE, s, "route",
                            [&] { return launch_route_shared(p, *shared_fp, d->w_dtype, s); });
    return timed_launch(CAEE_KERNEL_ROUTE, s, "route", [&] { return launch_route(p, s); });
}

int device_cu_count() {
    static int cached[64] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    if (!cached[dev]) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
        cached[dev] = n;
    }
    return cached[dev];
}

}  // namespace caee

namespace caee {
namespace {
caee_status_t check_layer_args(const caee_layer_desc_t* desc, const void* x, const float* logits, const float* bias,
                               const float* cost, const int32_t* bin, const caee_expert_weights_t* weights,
                               const void* y, const caee_route_out_t* out) {
    CAEE_TRY(check_desc(desc));
    CAEE_TRY(check_ptr(x, "x", true));
    CAEE_TRY(check_route_inputs(desc, logits, bias, cost, bin));
    if (out) CAEE_TRY(check_route_out(out));
    CAEE_TRY(check_weights(desc, weights));
    CAEE_TRY(check_ptr(y, "y", true));
    return CAEE_OK;
}

// The whole layer on validated arguments and a checked workspace; the big
// chunks run on a second stream when `side` is set.
caee_status_t moe_layer_run(const caee_layer_desc_t* desc, const void* x, const float* logits, const float* bias,
                            const float* cost, const int32_t* bin, const caee_expert_weights_t* weights, void* y,
                            const caee_route_out_t* out, char* wsb, const WsLayout& L, hipStream_t s, bool side) {
    RouteParams p = make_route_params(desc, logits, bias, cost, bin, wsb, L);
    p.chunk_big = call_chunk_big(*desc, weights->layout == CAEE_LAYOUT_TILED);
    set_route_outputs(p, out, wsb, L);
    const FfnParams fp = make_ffn_params(desc, x, p.topk_ids, p.topk_w, weights, y, wsb, L);
    FfnCall call;
    CAEE_TRY(ffn_begin(desc, fp, L, s, &call));
    call.shared_done = route_runs_shared(*desc);
    CAEE_TRY(run_route_layer(desc, p, out, wsb, L, s, call.shared_done ? &fp : nullptr));
    CAEE_TRY(ffn_routed(desc, fp, L, &call, side));
    return ffn_end(fp, &call);
}

// Scratch space of caee_moe_layer_noalloc: one array per GPU (each device
// holds its own copy at its own address), never freed.  In host code the
// array's name is not a device address; every host use goes through the
// address hipGetSymbolAddress returns for the current device.
__device__ __align__(256) unsigned char scratch[CAEE_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_at[kMaxDevices] = {};

caee_status_t scratch_address(void** at) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
        return fail(CAEE_ERR_HIP, "hipGetDevice failed or device index out of range");
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_at[dev]) {
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return fail(CAEE_ERR_HIP, "hipGetSymbolAddress of the scratch array failed: %s", hipGetErrorString(e));
        g_scratch_at[dev] = p;
    }
    *at = g_scratch_at[dev];
    return CAEE_OK;
}

struct NoTimingScope {
    NoTimingScope() { g_no_timing = true; }
    ~NoTimingScope() { g_no_timing = false; }
};
}  // namespace
}  // namespace caee

using namespace caee;

extern "C" {

caee_status_t caee_workspace_size(const caee_layer_desc_t* desc, size_t* bytes) {
    g_last_error.clear();
    if (!bytes) return fail(CAEE_ERR_INVALID_ARG, "bytes is NULL");
    CAEE_TRY(check_desc(desc));
    *bytes = ws_layout(*desc).total;
    return CAEE_OK;
}

caee_status_t caee_route_prune(const caee_layer_desc_t* desc, const float* logits, const float* bias,
                               const float* cost, const int32_t* bin, const caee_route_out_t* out, void* ws,
                               size_t ws_bytes, void* stream) {
    g_last_error.clear();
    CAEE_TRY(check_desc(desc));
    CAEE_TRY(check_route_inputs(desc, logits, bias, cost, bin));
    CAEE_TRY(check_route_out(out));
    WsLayout L;
    CAEE_TRY(check_ws(desc, ws, ws_bytes, &L));
    if (desc->T == 0) return CAEE_OK;
    RouteParams p = make_route_params(desc, logits, bias, cost, bin, (char*)ws, L);
    p.topk_ids = out->topk_ids;
    p.topk_w = out->topk_w;
    if (out->orig_ids) p.orig_ids = out->orig_ids;
    p.masks = out->masks;
    p.stats = out->stats;
    p.bin_loads = out->bin_loads;
    p.do_permute = 0;
    hipStream_t s = as_stream(stream);
    return timed_launch(CAEE_KERNEL_ROUTE, s, "route", [&] { return launch_route(p, s); });
}

caee_status_t caee_expert_ffn(const caee_layer_desc_t* desc, const void* x, const int32_t* topk_ids,
                              const float* topk_w, const caee_expert_weights_t* weights, void* y, void* ws,
                              size_t ws_bytes, void* stream) {
    g_last_error.clear();
    CAEE_TRY(check_desc(desc));
    CAEE_TRY(check_ptr(x, "x", true));
    CAEE_TRY(check_ptr(topk_ids, "topk_ids", true));
    CAEE_TRY(check_ptr(topk_w, "topk_w", true));
    CAEE_TRY(check_weights(desc, weights));
    CAEE_TRY(check_ptr(y, "y", true));
    WsLayout L;
    CAEE_TRY(check_ws(desc, ws, ws_bytes, &L));
    if (desc->T == 0) return CAEE_OK;
    RouteParams p = make_route_params(desc, nullptr, nullptr, nullptr, nullptr, (char*)ws, L);
    p.chunk_big = call_chunk_big(*desc, weights->layout == CAEE_LAYOUT_TILED);
    p.topk_ids = const_cast<int32_t*>(topk_ids);
    p.do_permute = 1;
    hipStream_t s = as_stream(stream);
    const FfnParams fp = make_ffn_params(desc, x, topk_ids, topk_w, weights, y, (char*)ws, L);
    FfnCall call;
    CAEE_TRY(ffn_begin(desc, fp, L, s, &call));
    CAEE_TRY(timed_launch(CAEE_KERNEL_ROUTE, s, "permute", [&] { return launch_permute(p, s); }));
    CAEE_TRY(ffn_routed(desc, fp, L, &call, true));
    return ffn_end(fp, &call);
}

caee_status_t caee_moe_layer(const caee_layer_desc_t* desc, const void* x, const float* logits, const float* bias,
                             const float* cost, const int32_t* bin, const caee_expert_weights_t* weights, void* y,
                             const caee_route_out_t* out, void* ws, size_t ws_bytes, void* stream) {
    g_last_error.clear();
    CAEE_TRY(check_layer_args(desc, x, logits, bias, cost, bin, weights, y, out));
    WsLayout L;
    CAEE_TRY(check_ws(desc, ws, ws_bytes, &L));
    if (desc->T == 0) return CAEE_OK;
    return moe_layer_run(desc, x, logits, bias, cost, bin, weights, y, out, (char*)ws, L, as_stream(stream), true);
}

caee_status_t caee_moe_layer_noalloc(const caee_layer_desc_t* desc, const void* x, const float* logits,
                                     const float* bias, const float* cost, const int32_t* bin,
                                     const caee_expert_weights_t* weights, void* y, const caee_route_out_t* out,
                                     void* stream) {
    g_last_error.clear();
    CAEE_TRY(check_layer_args(desc, x, logits, bias, cost, bin, weights, y, out));
    const WsLayout L = ws_layout(*desc);
    if (L.total > (size_t)CAEE_SCRATCH_BYTES)
        return fail(CAEE_ERR_UNSUPPORTED, "the call needs %zu bytes of scratch; the library's array holds %zu "
                    "(use caee_moe_layer with a workspace)", L.total, (size_t)CAEE_SCRATCH_BYTES);
    if (desc->T == 0) return CAEE_OK;
    void* at = nullptr;
    CAEE_TRY(scratch_address(&at));
    NoTimingScope no_timing;
    return moe_layer_run(desc, x, logits, bias, cost, bin, weights, y, out, (char*)at, L, as_stream(stream), false);
}

caee_status_t caee_pack_matrix(int32_t w_dtype, const void* src, void* dst, int64_t rows, int64_t cols,
                               int64_t count, void* stream) {
    g_last_error.clear();
    if (w_dtype != CAEE_F32 && w_dtype != CAEE_BF16 && w_dtype != CAEE_FP8_E4M3)
        return fail(CAEE_ERR_INVALID_ARG, "unknown w_dtype=%d", w_dtype);
    if (rows <= 0 || rows % 16) return fail(CAEE_ERR_INVALID_ARG, "rows=%lld must be a positive multiple of 16",
                                            (long long)rows);
    const long long row_bytes = (long long)cols * elem_bytes(w_dtype);
    if (cols <= 0 || row_bytes % 64)
        return fail(CAEE_ERR_INVALID_ARG, "a row (%lld bytes) must be a positive multiple of 64 bytes", row_bytes);
    if (count < 0) return fail(CAEE_ERR_INVALID_ARG, "count=%lld must be >= 0", (long long)count);
    CAEE_TRY(check_ptr(src, "src", true));
    CAEE_TRY(check_ptr(dst, "dst", true));
    const unsigned long long bytes = (unsigned long long)count * rows * row_bytes;
    const uintptr_t a = (uintptr_t)src, b = (uintptr_t)dst;
    if (a < b + bytes && b < a + bytes && bytes > 0) return fail(CAEE_ERR_INVALID_ARG, "src and dst overlap");
    if (count == 0) return CAEE_OK;
    const hipError_t err = launch_pack(src, dst, rows, row_bytes / 16, count, as_stream(stream));
    if (err != hipSuccess) return fail(CAEE_ERR_HIP, "pack launch failed: %s", hipGetErrorString(err));
    return CAEE_OK;
}

caee_status_t caee_quantize_rows(int32_t src_dtype, const void* src, int64_t rows, int64_t cols, uint8_t* q,
                                 float* scale, void* stream) {
    g_last_error.clear();
    if (src_dtype != CAEE_BF16 && src_dtype != CAEE_F32)
        return fail(CAEE_ERR_INVALID_ARG, "src_dtype=%d must be CAEE_BF16 or CAEE_F32", src_dtype);
    if (rows < 0 || cols <= 0 || cols % 128)
        return fail(CAEE_ERR_INVALID_ARG, "rows=%lld must be >= 0 and cols=%lld a positive multiple of 128",
                    (long long)rows, (long long)cols);
    CAEE_TRY(check_ptr(src, "src", true));
    CAEE_TRY(check_ptr(q, "q", true));
    CAEE_TRY(check_ptr(scale, "scale", true));
    if (rows == 0) return CAEE_OK;
    const hipError_t err =
        launch_quant_rows(src, src_dtype == CAEE_BF16, rows, (int)cols, q, scale, as_stream(stream));
    if (err != hipSuccess) return fail(CAEE_ERR_HIP, "quantise launch failed: %s", hipGetErrorString(err));
    return CAEE_OK;
}

const char* caee_status_str(caee_status_t status) {
    switch (status) {
        case CAEE_OK: return "ok";
        case CAEE_ERR_INVALID_ARG: return "invalid argument";
        case CAEE_ERR_UNSUPPORTED: return "unsupported by this build";
        case CAEE_ERR_WORKSPACE: return "workspace missing or too small";
        case CAEE_ERR_HIP: return "HIP runtime error";
        case CAEE_ERR_CAPACITY: return "more device slots needed than given";
    }
    return "unknown status";
}

const char* caee_last_error(void) { return g_last_error.c_str(); }

int caee_abi_version(void) { return CAEE_ABI_VERSION; }

caee_status_t caee_timing_enable(int on) {
    timing().on = on != 0;
    return CAEE_OK;
}

caee_status_t caee_timing_reset(void) {
    Timing& tm = timing();
    for (auto& r : tm.pending) {
        (void)hipEventSynchronize(r.b);
        tm.pool.push_back(r.a);
        tm.pool.push_back(r.b);
    }
    tm.pending.clear();
    for (int i = 0; i < CAEE_KERNEL_KINDS; ++i) {
        tm.total_ms[i] = 0.0;
        tm.launches[i] = 0;
    }
    return CAEE_OK;
}

caee_status_t caee_timing_query(int kind, double* total_ms, int64_t* launches) {
    g_last_error.clear();
    if (kind < 0 || kind >= CAEE_KERNEL_KINDS) return fail(CAEE_ERR_INVALID_ARG, "kind=%d out of range", kind);
    if (!total_ms || !launches) return fail(CAEE_ERR_INVALID_ARG, "NULL output pointer");
    Timing& tm = timing();
    for (auto& r : tm.pending) {
        if (hipEventSynchronize(r.b) != hipSuccess) return fail(CAEE_ERR_HIP, "hipEventSynchronize failed");
        float ms = 0.f;
        if (hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess) return fail(CAEE_ERR_HIP, "hipEventElapsedTime failed");
        tm.total_ms[r.kind] += ms;
        tm.launches[r.kind] += 1;
        tm.pool.push_back(r.a);
        tm.pool.push_back(r.b);
    }
    tm.pending.clear();
    *total_ms = tm.total_ms[kind];
    *launches = tm.launches[kind];
    return CAEE_OK;
}

}  // extern "C"
