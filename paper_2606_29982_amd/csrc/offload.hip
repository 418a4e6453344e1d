// Offload residency for the offloading deployment (Sec. V-B): routed experts
// live in page-locked host memory, a bounded set of them in device cache
// slots.  Host code only; the FFN kernels take each expert's weight address
// from a per-call pointer table and run in passes, so that the experts
// already on the device compute while the missing ones are still being
// copied over the host link.
//
// Per call:  cost table from residency (Sec. IV-A: R = 0 for a resident
// expert) -> routing/pruning/compensation on `stream` -> host reads A_trans
// -> LRU plan -> H2D copies in batches on `copy_stream` -> FFN pass of the
// hits, then one pass per batch as it lands -> combine.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <vector>

#include "caee_internal.h"

using namespace caee;

struct caee_offload {
    caee_layer_desc_t desc{};
    int device = 0;
    std::vector<const void*> host_w13, host_w2;
    char* slot_w13 = nullptr;
    char* slot_w2 = nullptr;
    const char* sh_w13 = nullptr;
    const char* sh_w2 = nullptr;
    int layout = 0, n_cache = 0, n_stage = 0, fetch_batch = 1;
    float miss_cost = 1.0f;
    size_t w13_bytes = 0, w2_bytes = 0;      // one expert
    // residency
    std::vector<int32_t> slot_of, slot_expert;
    std::vector<int64_t> slot_used;
    int64_t call = 0;
    caee_offload_stats_t st{};
    // per-call tables: device block and its page-locked host mirror
    //   cost [E] fp32 | wtab [2 (E + n_shared)] pointers | pass_of [E + n_shared] int32
    char* dev_tab = nullptr;
    char* host_tab = nullptr;
    size_t off_wtab = 0, off_pass = 0, tab_bytes = 0;
    uint8_t* host_trans = nullptr;           // [E] A_trans flags read back after routing
    hipEvent_t ev_route = nullptr, ev_done = nullptr;
    bool have_done = false;
    std::vector<hipEvent_t> ev_fetch, ev_pass;
};

namespace {

size_t align256_(size_t v) { return (v + 255) & ~size_t(255); }

caee_status_t hip_fail(hipError_t e, const char* what) {
    return fail(CAEE_ERR_HIP, "%s failed: %s", what, hipGetErrorString(e));
}

#define HIP_TRY(expr, what)                          \
    do {                                             \
        hipError_t e_ = (expr);                      \
        if (e_ != hipSuccess) return hip_fail(e_, what); \
    } while (0)

bool page_locked(const void* p) {
    hipPointerAttribute_t a;
    if (hipPointerGetAttributes(&a, p) != hipSuccess) {
        (void)hipGetLastError();   // the query sets the last error for unknown (pageable) pointers
        return false;
    }
    return a.type == hipMemoryTypeHost;
}

caee_status_t lru_plan(int E, int n_cache, int n_stage, int32_t* slot_of, int32_t* slot_expert, int64_t* slot_used,
                       int64_t call, const uint8_t* need, int32_t* fetch, int32_t* fetch_slot, int32_t* counts) {
    for (int e = 0; e < E; ++e) {
        const int s = slot_of[e];
        if (s < -1 || s >= n_cache || (s >= 0 && slot_expert[s] != e))
            return fail(CAEE_ERR_INVALID_ARG, "slot_of[%d]=%d is inconsistent with slot_expert", e, s);
    }
    for (int i = 0; i < n_cache; ++i) {
        const int e = slot_expert[i];
        if (e < -1 || e >= E || (e >= 0 && slot_of[e] != i))
            return fail(CAEE_ERR_INVALID_ARG, "slot_expert[%d]=%d is inconsistent with slot_of", i, e);
        if (e >= 0 && slot_used[i] >= call)
            return fail(CAEE_ERR_INVALID_ARG, "slot_used[%d]=%lld is not before call %lld", i,
                        (long long)slot_used[i], (long long)call);
    }
    int hits = 0, misses = 0;
    for (int e = 0; e < E; ++e)
        if (need[e]) (slot_of[e] >= 0 ? hits : misses) += 1;
    // Slots a miss may take: empty ones first (lowest index), then those whose
    // expert this call does not need, least recently used first.
    std::vector<int> avail, victims;
    for (int i = 0; i < n_cache; ++i) {
        if (slot_expert[i] < 0)
            avail.push_back(i);
        else if (!need[slot_expert[i]])
            victims.push_back(i);
    }
    std::sort(victims.begin(), victims.end(), [&](int a, int b) {
        if (slot_used[a] != slot_used[b]) return slot_used[a] < slot_used[b];
        return slot_expert[a] < slot_expert[b];
    });
    avail.insert(avail.end(), victims.begin(), victims.end());
    const int cached = std::min<int>(misses, (int)avail.size());
    const int staged = misses - cached;
    if (staged > 0 && n_stage <= 0)
        return fail(CAEE_ERR_CAPACITY, "%d misses but only %d cache slots free and no staging slots", misses, cached);
    int n = 0, evictions = 0;
    for (int e = 0; e < E; ++e) {
        if (!need[e] || slot_of[e] >= 0) continue;
        if (n < cached) {
            const int s = avail[n];
            if (slot_expert[s] >= 0) {
                slot_of[slot_expert[s]] = -1;
                ++evictions;
            }
            slot_expert[s] = e;
            slot_of[e] = s;
            fetch_slot[n] = s;
        } else {
            fetch_slot[n] = n_cache + (n - cached) % n_stage;
        }
        fetch[n++] = e;
    }
    for (int e = 0; e < E; ++e)
        if (need[e] && slot_of[e] >= 0) slot_used[slot_of[e]] = call;
    counts[0] = hits;
    counts[1] = misses;
    counts[2] = staged;
    counts[3] = evictions;
    return CAEE_OK;
}

caee_status_t ensure_events(std::vector<hipEvent_t>& v, size_t n) {
    while (v.size() < n) {
        hipEvent_t e = nullptr;
        HIP_TRY(hipEventCreateWithFlags(&e, hipEventDisableTiming), "hipEventCreateWithFlags");
        v.push_back(e);
    }
    return CAEE_OK;
}

void release(caee_offload* h) {
    if (!h) return;
    if (h->ev_done && h->have_done) (void)hipEventSynchronize(h->ev_done);
    if (h->dev_tab) (void)hipFree(h->dev_tab);
    if (h->host_tab) (void)hipHostFree(h->host_tab);
    if (h->host_trans) (void)hipHostFree(h->host_trans);
    if (h->ev_route) (void)hipEventDestroy(h->ev_route);
    if (h->ev_done) (void)hipEventDestroy(h->ev_done);
    for (auto e : h->ev_fetch) (void)hipEventDestroy(e);
    for (auto e : h->ev_pass) (void)hipEventDestroy(e);
    delete h;
}

caee_status_t wait_idle(caee_offload* h) {
    if (h->have_done) HIP_TRY(hipEventSynchronize(h->ev_done), "hipEventSynchronize");
    return CAEE_OK;
}

}  // namespace

extern "C" {

caee_status_t caee_lru_step(int32_t E, int32_t n_cache, int32_t n_stage, int32_t* slot_of, int32_t* slot_expert,
                            int64_t* slot_used, int64_t call, const uint8_t* need, int32_t* fetch,
                            int32_t* fetch_slot, int32_t* counts) {
    clear_last_error();
    if (E < 1 || E > kMaxE) return fail(CAEE_ERR_INVALID_ARG, "E=%d must be in [1, %d]", E, kMaxE);
    if (n_cache < 0 || n_stage < 0 || n_cache + n_stage < 1)
        return fail(CAEE_ERR_INVALID_ARG, "n_cache=%d, n_stage=%d: both >= 0 and at least one slot", n_cache, n_stage);
    if (!slot_of || !need || !fetch || !fetch_slot || !counts || (n_cache > 0 && (!slot_expert || !slot_used)))
        return fail(CAEE_ERR_INVALID_ARG, "NULL array");
    return lru_plan(E, n_cache, n_stage, slot_of, slot_expert, slot_used, call, need, fetch, fetch_slot, counts);
}

caee_status_t caee_offload_create(const caee_layer_desc_t* desc, const caee_offload_desc_t* od,
                                  caee_offload_t** handle) {
    clear_last_error();
    if (!handle) return fail(CAEE_ERR_INVALID_ARG, "handle is NULL");
    *handle = nullptr;
    caee_layer_desc_t d0;
    if (!desc) return fail(CAEE_ERR_INVALID_ARG, "desc is NULL");
    d0 = *desc;
    d0.T = 0;
    CAEE_TRY(check_desc(&d0));
    if (!od) return fail(CAEE_ERR_INVALID_ARG, "offload desc is NULL");
    if (d0.w_dtype != CAEE_BF16 && d0.w_dtype != CAEE_F32)
        return fail(CAEE_ERR_UNSUPPORTED, "offload supports CAEE_BF16 and CAEE_F32 weights");
    if (od->layout != CAEE_LAYOUT_ROWMAJOR && od->layout != CAEE_LAYOUT_TILED)
        return fail(CAEE_ERR_INVALID_ARG, "unknown weight layout=%d", od->layout);
    if (od->n_cache < 0 || od->n_stage < 0 || od->n_cache + od->n_stage < 1)
        return fail(CAEE_ERR_INVALID_ARG, "n_cache=%d, n_stage=%d: both >= 0 and at least one slot", od->n_cache,
                    od->n_stage);
    if (od->fetch_batch < 1) return fail(CAEE_ERR_INVALID_ARG, "fetch_batch=%d must be >= 1", od->fetch_batch);
    if (!(std::isfinite(od->miss_cost) && od->miss_cost > 0.0f))
        return fail(CAEE_ERR_INVALID_ARG, "miss_cost must be finite and > 0");
    if (!od->host_w13 || !od->host_w2) return fail(CAEE_ERR_INVALID_ARG, "host pointer arrays are NULL");
    CAEE_TRY(check_ptr(od->slot_w13, "slot_w13", true));
    CAEE_TRY(check_ptr(od->slot_w2, "slot_w2", true));
    const bool sh = d0.n_shared > 0;
    CAEE_TRY(check_ptr(od->sh_w13, "sh_w13", sh));
    CAEE_TRY(check_ptr(od->sh_w2, "sh_w2", sh));
    if (!sh && (od->sh_w13 || od->sh_w2)) return fail(CAEE_ERR_INVALID_ARG, "shared weights given with n_shared=0");
    for (int e = 0; e < d0.E; ++e) {
        CAEE_TRY(check_ptr(od->host_w13[e], "host_w13[e]", true));
        CAEE_TRY(check_ptr(od->host_w2[e], "host_w2[e]", true));
        if (!page_locked(od->host_w13[e]) || !page_locked(od->host_w2[e]))
            return fail(CAEE_ERR_INVALID_ARG, "host weights of expert %d are not page-locked host memory", e);
    }
    caee_offload* h = new caee_offload();
    h->desc = d0;
    if (hipGetDevice(&h->device) != hipSuccess) {
        release(h);
        return fail(CAEE_ERR_HIP, "hipGetDevice failed");
    }
    h->host_w13.assign(od->host_w13, od->host_w13 + d0.E);
    h->host_w2.assign(od->host_w2, od->host_w2 + d0.E);
    h->slot_w13 = (char*)od->slot_w13;
    h->slot_w2 = (char*)od->slot_w2;
    h->sh_w13 = (const char*)od->sh_w13;
    h->sh_w2 = (const char*)od->sh_w2;
    h->layout = od->layout;
    h->n_cache = od->n_cache;
    h->n_stage = od->n_stage;
    h->fetch_batch = od->fetch_batch;
    h->miss_cost = od->miss_cost;
    const size_t eb = elem_bytes(d0.w_dtype);
    h->w13_bytes = (size_t)2 * d0.f * d0.d * eb;
    h->w2_bytes = (size_t)d0.d * d0.f * eb;
    h->slot_of.assign(d0.E, -1);
    h->slot_expert.assign(h->n_cache, -1);
    h->slot_used.assign(h->n_cache, -1);
    const int X = d0.E + d0.n_shared;
    h->off_wtab = align256_((size_t)d0.E * 4);
    h->off_pass = h->off_wtab + align256_((size_t)2 * X * sizeof(void*));
    h->tab_bytes = h->off_pass + align256_((size_t)X * 4);
    hipError_t e1 = hipMalloc((void**)&h->dev_tab, h->tab_bytes);
    hipError_t e2 = e1 == hipSuccess ? hipHostMalloc((void**)&h->host_tab, h->tab_bytes, hipHostMallocDefault) : e1;
    hipError_t e3 = e2 == hipSuccess ? hipHostMalloc((void**)&h->host_trans, align256_(d0.E), hipHostMallocDefault) : e2;
    hipError_t e4 = e3 == hipSuccess ? hipEventCreateWithFlags(&h->ev_route, hipEventDisableTiming) : e3;
    hipError_t e5 = e4 == hipSuccess ? hipEventCreateWithFlags(&h->ev_done, hipEventDisableTiming) : e4;
    if (e5 != hipSuccess) {
        release(h);
        return hip_fail(e5, "offload allocation");
    }
    std::memset(h->host_tab, 0, h->tab_bytes);
    *handle = h;
    return CAEE_OK;
}

void caee_offload_destroy(caee_offload_t* handle) { release(handle); }

caee_status_t caee_offload_stats(const caee_offload_t* h, caee_offload_stats_t* stats) {
    clear_last_error();
    if (!h || !stats) return fail(CAEE_ERR_INVALID_ARG, "NULL argument");
    *stats = h->st;
    return CAEE_OK;
}

caee_status_t caee_offload_residency(const caee_offload_t* h, int32_t* slot_of) {
    clear_last_error();
    if (!h || !slot_of) return fail(CAEE_ERR_INVALID_ARG, "NULL argument");
    std::copy(h->slot_of.begin(), h->slot_of.end(), slot_of);
    return CAEE_OK;
}

caee_status_t caee_offload_reset(caee_offload_t* h) {
    clear_last_error();
    if (!h) return fail(CAEE_ERR_INVALID_ARG, "handle is NULL");
    CAEE_TRY(wait_idle(h));
    std::fill(h->slot_of.begin(), h->slot_of.end(), -1);
    std::fill(h->slot_expert.begin(), h->slot_expert.end(), -1);
    std::fill(h->slot_used.begin(), h->slot_used.end(), -1);
    h->call = 0;
    h->st = caee_offload_stats_t{};
    return CAEE_OK;
}

caee_status_t caee_offload_layer(caee_offload_t* h, const caee_layer_desc_t* desc, const void* x,
                                 const float* logits, const float* bias, void* y, const caee_route_out_t* out,
                                 void* ws, size_t ws_bytes, void* stream, void* copy_stream) {
    clear_last_error();
    if (!h) return fail(CAEE_ERR_INVALID_ARG, "handle is NULL");
    CAEE_TRY(check_desc(desc));
    const caee_layer_desc_t& d = *desc;
    if (d.d != h->desc.d || d.f != h->desc.f || d.E != h->desc.E || d.n_shared != h->desc.n_shared ||
        d.w_dtype != h->desc.w_dtype)
        return fail(CAEE_ERR_INVALID_ARG, "desc does not match the handle's layer (d, f, E, n_shared, w_dtype)");
    if (d.n_bins != 1) return fail(CAEE_ERR_INVALID_ARG, "offload calls take n_bins=1 (one host link)");
    CAEE_TRY(check_ptr(x, "x", true));
    CAEE_TRY(check_ptr(logits, "logits", true));
    CAEE_TRY(check_ptr(bias, "bias", false));
    if (out) CAEE_TRY(check_route_out(out));
    CAEE_TRY(check_ptr(y, "y", true));
    WsLayout L;
    CAEE_TRY(check_ws(desc, ws, ws_bytes, &L));
    int dev = -1;
    HIP_TRY(hipGetDevice(&dev), "hipGetDevice");
    if (dev != h->device) return fail(CAEE_ERR_INVALID_ARG, "current device %d is not the handle's %d", dev, h->device);
    if (d.T == 0) return CAEE_OK;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    hipStream_t cs = reinterpret_cast<hipStream_t>(copy_stream);
    char* wsb = (char*)ws;
    const int E = d.E, X = d.E + d.n_shared;

    // Tables and slots are rewritten below; the previous call must be done with them.
    if (h->have_done) HIP_TRY(hipStreamWaitEvent(s, h->ev_done, 0), "hipStreamWaitEvent");
    // 1. cost table from residency, then routing with one bin.
    float* hcost = (float*)h->host_tab;
    for (int e = 0; e < E; ++e) hcost[e] = h->slot_of[e] >= 0 ? 0.0f : h->miss_cost;
    HIP_TRY(hipMemcpyAsync(h->dev_tab, hcost, (size_t)E * 4, hipMemcpyHostToDevice, s), "cost table copy");
    RouteParams rp = make_route_params(desc, logits, bias, (const float*)h->dev_tab, nullptr, wsb, L);
    rp.chunk_big = call_chunk_big(d, h->layout == CAEE_LAYOUT_TILED);
    set_route_outputs(rp, out, wsb, L);
    FfnParams fp = make_ffn_params(desc, x, rp.topk_ids, rp.topk_w, nullptr, y, wsb, L);
    fp.sh_w13 = h->sh_w13;
    fp.sh_w2 = h->sh_w2;
    fp.tiled = h->layout == CAEE_LAYOUT_TILED;
    fp.wtab = (const void* const*)(h->dev_tab + h->off_wtab);
    fp.pass_of = (const int32_t*)(h->dev_tab + h->off_pass);
    fp.pass_id = 0;
    FfnCall fc;
    CAEE_TRY(ffn_begin(desc, fp, L, s, &fc));
    // Any return below must first bring the side stream back into `stream`.
    auto joined = [&](caee_status_t st) {
        if (fc.side != fc.main && hipEventRecord(fc.ev_join, fc.side) == hipSuccess)
            (void)hipStreamWaitEvent(fc.main, fc.ev_join, 0);
        return st;
    };
    fc.shared_done = route_runs_shared(d);   // as caee_moe_layer, so both give the same bits
    caee_status_t st = run_route_layer(desc, rp, out, wsb, L, s, fc.shared_done ? &fp : nullptr);
    if (st != CAEE_OK) return joined(st);
    // 2. read A_trans back.
    hipError_t he = hipMemcpyAsync(h->host_trans, wsb + L.trans, E, hipMemcpyDeviceToHost, s);
    if (he == hipSuccess) he = hipEventRecord(h->ev_route, s);
    if (he == hipSuccess) he = hipEventSynchronize(h->ev_route);
    if (he != hipSuccess) return joined(hip_fail(he, "A_trans read-back"));

    // 3. plan.
    std::vector<int32_t> fetch(E), fetch_slot(E);
    int32_t counts[4];
    const int64_t call = h->call;
    st = lru_plan(E, h->n_cache, h->n_stage, h->slot_of.data(), h->slot_expert.data(), h->slot_used.data(), call,
                  h->host_trans, fetch.data(), fetch_slot.data(), counts);
    if (st != CAEE_OK) return joined(st);
    const int misses = counts[1], staged = counts[2];
    const int batch = staged > 0 ? std::min(h->fetch_batch, h->n_stage) : h->fetch_batch;
    const int n_batches = (misses + batch - 1) / batch;
    // Undo the residency of this call's cached misses if anything below fails.
    auto rollback = [&](caee_status_t st_) {
        for (int i = 0; i < misses - staged; ++i) {
            const int sl = fetch_slot[i];
            h->slot_of[fetch[i]] = -1;
            h->slot_expert[sl] = -1;
            h->slot_used[sl] = -1;
        }
        return joined(st_);
    };

    // Tables: weight addresses and the pass of every expert slot.
    const void** wtab = (const void**)(h->host_tab + h->off_wtab);
    int32_t* pass_of = (int32_t*)(h->host_tab + h->off_pass);
    for (int e = 0; e < E; ++e) {
        const int sl = h->slot_of[e] >= 0 && h->host_trans[e] ? h->slot_of[e] : 0;
        wtab[2 * e] = h->slot_w13 + (size_t)sl * h->w13_bytes;
        wtab[2 * e + 1] = h->slot_w2 + (size_t)sl * h->w2_bytes;
        pass_of[e] = h->host_trans[e] ? 0 : -1;
    }
    for (int i = 0; i < misses; ++i) {
        const int e = fetch[i], sl = fetch_slot[i];
        wtab[2 * e] = h->slot_w13 + (size_t)sl * h->w13_bytes;
        wtab[2 * e + 1] = h->slot_w2 + (size_t)sl * h->w2_bytes;
        pass_of[e] = 1 + i / batch;
    }
    for (int sx = 0; sx < d.n_shared; ++sx) {
        wtab[2 * (E + sx)] = h->sh_w13 + (size_t)sx * h->w13_bytes;
        wtab[2 * (E + sx) + 1] = h->sh_w2 + (size_t)sx * h->w2_bytes;
        pass_of[E + sx] = 0;
    }
    (void)X;
    if (ensure_events(h->ev_fetch, n_batches) != CAEE_OK || ensure_events(h->ev_pass, n_batches + 1) != CAEE_OK)
        return rollback(CAEE_ERR_HIP);
    he = hipMemcpyAsync(h->dev_tab + h->off_wtab, h->host_tab + h->off_wtab, h->tab_bytes - h->off_wtab,
                        hipMemcpyHostToDevice, s);
    if (he != hipSuccess) return rollback(hip_fail(he, "table copy"));

    // 4. copies and FFN passes.  Slots overwritten here were last read by an
    // earlier call, which ended with ev_done.
    if (misses > 0 && h->have_done) {
        he = hipStreamWaitEvent(cs, h->ev_done, 0);
        if (he != hipSuccess) return rollback(hip_fail(he, "hipStreamWaitEvent"));
    }
    st = ffn_routed(desc, fp, L, &fc, false);
    if (st != CAEE_OK) return rollback(st);
    const int cached = misses - staged;
    for (int b = 0; b < n_batches; ++b) {
        for (int i = b * batch; i < std::min(misses, (b + 1) * batch); ++i) {
            const int q = i - cached;   // staging index (< 0: a cache slot)
            if (q >= h->n_stage) {
                // The staging slot's previous occupant (miss i - n_stage) must have been computed.
                he = hipStreamWaitEvent(cs, h->ev_pass[1 + (i - h->n_stage) / batch], 0);
                if (he != hipSuccess) return rollback(hip_fail(he, "hipStreamWaitEvent"));
            }
            const int e = fetch[i], sl = fetch_slot[i];
            he = hipMemcpyAsync(h->slot_w13 + (size_t)sl * h->w13_bytes, h->host_w13[e], h->w13_bytes,
                                hipMemcpyHostToDevice, cs);
            if (he == hipSuccess)
                he = hipMemcpyAsync(h->slot_w2 + (size_t)sl * h->w2_bytes, h->host_w2[e], h->w2_bytes,
                                    hipMemcpyHostToDevice, cs);
            if (he != hipSuccess) return rollback(hip_fail(he, "expert copy"));
        }
        he = hipEventRecord(h->ev_fetch[b], cs);
        if (he == hipSuccess) he = hipStreamWaitEvent(s, h->ev_fetch[b], 0);
        if (he != hipSuccess) return rollback(hip_fail(he, "fetch event"));
        fp.pass_id = 1 + b;
        st = ffn_routed(desc, fp, L, &fc, false);
        if (st != CAEE_OK) return rollback(st);
        he = hipEventRecord(h->ev_pass[1 + b], s);
        if (he != hipSuccess) return rollback(hip_fail(he, "pass event"));
    }
    // 5. join and combine.
    st = ffn_end(fp, &fc);
    if (st != CAEE_OK) return rollback(st);
    he = hipEventRecord(h->ev_done, s);
    if (he != hipSuccess) return rollback(hip_fail(he, "hipEventRecord"));
    h->have_done = true;
    h->call = call + 1;
    h->st.calls += 1;
    h->st.needed += counts[0] + counts[1];
    h->st.hits += counts[0];
    h->st.misses += misses;
    h->st.staged += staged;
    h->st.evictions += counts[3];
    h->st.bytes_h2d += (int64_t)misses * (int64_t)(h->w13_bytes + h->w2_bytes);
    h->st.passes = 1 + n_batches;
    return CAEE_OK;
}

}  // extern "C"
