// Routing, cost-aware pruning, compensation and token permutation for one
// MoE layer call: token-parallel kernels, and for batches of up to 16 tokens
// one 1024-thread workgroup that runs every phase.
//
//   phase A (one wavefront per token): sigmoid scores, group-limited top-k
//            K_t and normalised gate weights G(t)_e (Sec. II-A);
//   phase B (whole workgroup): importance, mandatory/candidate split,
//            per-bin baseline cost F_base and cost-invariant expansion
//            (Sec. IV-A, IV-B steps 1-4);
//   phase C (one wavefront per token): masking of pruned experts and
//            top-k refill from A_trans (Sec. IV-C), weight renormalisation;
//   permute: stable counting sort of the (token, expert) pairs by expert,
//            the shared experts' rows first, and the FFN work lists (small
//            and big expert chunks).
//
// Every decision is taken in float64 with ties to the lower index, so the
// result does not depend on the order in which lanes or waves finish.
#include <math.h>

#include "caee_internal.h"

namespace caee {
namespace {

#include "ffn_tile.h"

constexpr int kTokWaves = 4;                       // tokens (wavefronts) per workgroup
constexpr int kTokThreads = kTokWaves * kWave;
// Batches up to this many tokens are routed by one fused single-workgroup kernel.
#ifndef CAEE_FUSED_T
#define CAEE_FUSED_T 16
#endif
constexpr int kFusedT = CAEE_FUSED_T;
constexpr int kNoIdx = 0x7fffffff;

// Cross-lane moves within a 16-lane row through DPP (no LDS round trip).
template <int C>
__device__ inline int dpp_i(int v) {
    return __builtin_amdgcn_mov_dpp(v, C, 0xF, 0xF, false);
}
template <int C>
__device__ inline double dpp_d(double v) {
    const long long b = __double_as_longlong(v);
    const int lo = dpp_i<C>((int)b);
    const int hi = dpp_i<C>((int)(b >> 32));
    return __longlong_as_double(((long long)hi << 32) | (unsigned int)lo);
}
__device__ inline double readlane_d(double v, int lane) {
    const long long b = __double_as_longlong(v);
    const int lo = __builtin_amdgcn_readlane((int)b, lane);
    const int hi = __builtin_amdgcn_readlane((int)(b >> 32), lane);
    return __longlong_as_double(((long long)hi << 32) | (unsigned int)lo);
}

// DPP controls that pair every lane of a row with another one:
// quad_perm [1,0,3,2], quad_perm [2,3,0,1], row_half_mirror, row_mirror.
constexpr int kDppXor1 = 0xB1, kDppXor2 = 0x4E, kDppHalfMirror = 0x141, kDppMirror = 0x140;


// Row broadcasts of gfx9 DPP: lane 15 of each row to the next row, lane 31
// to rows 2 and 3.  Rows outside `RM` keep their own value (update_dpp's
// old operand), so a max or min with it changes nothing there.
constexpr int kDppRowBcast15 = 0x142, kDppRowBcast31 = 0x143;
template <int C, int RM>
__device__ inline int dpp_upd_i(int v) {
    return __builtin_amdgcn_update_dpp(v, v, C, RM, 0xF, false);
}
template <int C, int RM>
__device__ inline double dpp_upd_d(double v) {
    const long long b = __double_as_longlong(v);
    const int lo = dpp_upd_i<C, RM>((int)b);
    const int hi = dpp_upd_i<C, RM>((int)(b >> 32));
    return __longlong_as_double(((long long)hi << 32) | (unsigned int)lo);
}

// Wave-wide max and min, all in VALU: butterfly inside each 16-lane row,
// then row 1 takes row 0's result and row 3 row 2's, then row 3 takes row
// 1's; lane 63 ends with the wave's result, which every lane reads.
__device__ inline double wave_max_d(double v) {
    v = fmax(v, dpp_d<kDppXor1>(v));
    v = fmax(v, dpp_d<kDppXor2>(v));
    v = fmax(v, dpp_d<kDppHalfMirror>(v));
    v = fmax(v, dpp_d<kDppMirror>(v));
    v = fmax(v, dpp_upd_d<kDppRowBcast15, 0xA>(v));
    v = fmax(v, dpp_upd_d<kDppRowBcast31, 0xC>(v));
    return readlane_d(v, 63);
}
__device__ inline int wave_min_i(int v) {
    v = min(v, dpp_i<kDppXor1>(v));
    v = min(v, dpp_i<kDppXor2>(v));
    v = min(v, dpp_i<kDppHalfMirror>(v));
    v = min(v, dpp_i<kDppMirror>(v));
    v = min(v, dpp_upd_i<kDppRowBcast15, 0xA>(v));
    v = min(v, dpp_upd_i<kDppRowBcast31, 0xC>(v));
    return __builtin_amdgcn_readlane(v, 63);
}

// Inclusive prefix sum over the 64 lanes, in VALU: shifts by 1, 2, 4, 8
// within each row (lanes shifted in from outside the row read 0), then
// rows 1 and 3 add the last lane of rows 0 and 2, rows 2 and 3 that of row 1.
__device__ inline int wave_incl_scan(int v) {
    v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, true);   // row_shr:1
    v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, true);   // row_shr:2
    v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, true);   // row_shr:4
    v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, true);   // row_shr:8
    v += __builtin_amdgcn_update_dpp(0, v, kDppRowBcast15, 0xA, 0xF, false);
    v += __builtin_amdgcn_update_dpp(0, v, kDppRowBcast31, 0xC, 0xF, false);
    return v;
}

// Wave-wide argmax of (v, i): the largest v, and among the lanes holding it
// the lowest i (the same result as merging pairs in any order).  Values are
// never NaN.  Every lane gets the result.
__device__ inline void wave_argmax(double& v, int& i) {
    const double m = wave_max_d(v);
    i = wave_min_i(v == m ? i : kNoIdx);
    v = m;
}

// Merge two (largest, second largest) pairs.
__device__ inline void top2_merge(double& t1, double& t2, double o1, double o2) {
    const double n1 = fmax(t1, o1);
    const double n2 = fmax(fmin(t1, o1), fmax(t2, o2));
    t1 = n1;
    t2 = n2;
}
template <int C>
__device__ inline void top2_step(double& t1, double& t2) {
    top2_merge(t1, t2, dpp_d<C>(t1), dpp_d<C>(t2));
}

// Lane `lane` holds experts lane*EPL .. lane*EPL+EPL-1.
template <int EPL>
__device__ inline void load_scores(const RouteParams& p, int t, int lane, double (&s)[EPL],
                                   double (&key)[EPL]) {
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
        const int e = lane * EPL + i;
        if (e < p.E) {
            const double z = (double)p.logits[(size_t)t * p.E + e];
            const double sv = 1.0 / (1.0 + exp(-z));
            s[i] = sv;
            key[i] = sv + (p.bias ? (double)p.bias[e] : 0.0);
        } else {
            s[i] = 0.0;
            key[i] = -INFINITY;
        }
    }
}

// Each lane's score s of expert `e` (its own, or 0 when `valid` is false),
// fetched from the lane that holds it: one shuffle per element slot, for all
// lanes at once.
template <int EPL>
__device__ inline double fetch_score(const double (&s)[EPL], int e, bool valid, int E) {
    const bool ok = valid && e >= 0 && e < E;
    const int src = ok ? e / EPL : 0;
    const int which = ok ? e % EPL : 0;
    double got = 0.0;
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
        const double c = __shfl(s[i], src);
        if (which == i) got = c;
    }
    return ok ? got : 0.0;
}

// Groups ranked in one pass (each lane reads every group's score) when
// there are at most this many; more groups take one wave argmax per pick.
constexpr int kRankGroups = 16;

// Phase A for token t: writes K_t (rank order), G(t) and the token's top expert.
template <int EPL>
__device__ void route_token(const RouteParams& p, int t, int lane, int* ids, double* gout,
                            int* top1, uint8_t* mflag) {
    double s[EPL], key[EPL];
    load_scores<EPL>(p, t, lane, s, key);
    const bool lane_valid = lane * EPL < p.E;

    // Group score: sum of the two largest keys of the group.
    double t1 = -INFINITY, t2 = -INFINITY;
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
        if (key[i] > t1) {
            t2 = t1;
            t1 = key[i];
        } else if (key[i] > t2) {
            t2 = key[i];
        }
    }
    // Reduce over the lpg lanes holding one group (aligned blocks of lpg lanes).
    if (p.lpg >= 2) top2_step<kDppXor1>(t1, t2);
    if (p.lpg >= 4) top2_step<kDppXor2>(t1, t2);
    if (p.lpg >= 8) top2_step<kDppHalfMirror>(t1, t2);
    if (p.lpg >= 16) top2_step<kDppMirror>(t1, t2);
    for (int off = 16; off < p.lpg; off <<= 1) top2_merge(t1, t2, __shfl_xor(t1, off), __shfl_xor(t2, off));
    const double gscore = p.gsize >= 2 ? t1 + t2 : t1;
    const int my_group = lane_valid ? (lane * EPL) / p.gsize : kNoIdx;

    bool gsel = false;
    if (p.n_group <= kRankGroups) {
        // The group's rank: groups with a larger score, or the same score and
        // a lower index, come first; the first topk_group are selected.
        int rank = 0;
        for (int g2 = 0; g2 < p.n_group; ++g2) {
            const double o = readlane_d(gscore, g2 * p.lpg);   // the group's first lane
            rank += (o > gscore) | ((o == gscore) & (g2 < my_group));
        }
        gsel = lane_valid && rank < p.topk_group;
    } else {
        for (int r = 0; r < p.topk_group; ++r) {
            double v = (lane_valid && !gsel) ? gscore : -INFINITY;
            int gi = (lane_valid && !gsel) ? my_group : kNoIdx;
            wave_argmax(v, gi);
            if (my_group == gi) gsel = true;
        }
    }

    // Top-k keys of the selected groups; lane r keeps the r-th pick.
    bool chosen[EPL];
#pragma unroll
    for (int i = 0; i < EPL; ++i) chosen[i] = false;
    int my_id = kNoIdx;
    double my_s = 0.0;
    for (int r = 0; r < p.k; ++r) {
        double v = -INFINITY;
        int ei = kNoIdx;
#pragma unroll
        for (int i = 0; i < EPL; ++i) {
            if (gsel && !chosen[i] && key[i] > v) {
                v = key[i];
                ei = lane * EPL + i;
            }
        }
        wave_argmax(v, ei);
#pragma unroll
        for (int i = 0; i < EPL; ++i)
            if (lane * EPL + i == ei) chosen[i] = true;
        if (lane == r) my_id = ei;
    }
    my_s = fetch_score<EPL>(s, my_id, lane < p.k, p.E);
    // G(t): each score over the token's k scores summed in rank order (the
    // same additions on every lane), one slot per lane.
    double total = 0.0;
    for (int r = 0; r < p.k; ++r) total += readlane_d(my_s, r);
    const bool mine = lane < p.k;
    const double g = my_s / total;
    double bg = mine ? g : -INFINITY;
    int best = mine ? my_id : kNoIdx;
    wave_argmax(bg, best);   // the token's top expert by G, ties to the lower index
    // Pairs that are mandatory on their own: the threshold (MAX) or the
    // cumulative-ratio prefix (CIR), and with keep_top1 the token's top expert.
    uint32_t flags = (uint32_t)__ballot(
        mine && ((p.keep_top1 && my_id == best) || (p.rule == CAEE_IMPORTANCE_MAX && g >= p.tau)));
    if (mine) {
        ids[lane] = my_id;
        gout[lane] = g;
        if (p.sslot) p.sslot[(size_t)t * p.k + lane] = my_s;
    }
    if (lane == 0) *top1 = best;
    if (p.rule == CAEE_IMPORTANCE_CIR) {
        // Slots in gate order (score descending, lower expert first on ties):
        // each slot's lane counts the slots ahead of it; the prefix then
        // walks the positions in order, the same additions on every lane.
        int ahead = 0;
        for (int j = 0; j < p.k; ++j) {
            const double sj = readlane_d(my_s, j);
            const int ij = __builtin_amdgcn_readlane(my_id, j);
            ahead += (sj > my_s || (sj == my_s && ij < my_id)) ? 1 : 0;
        }
        auto lane_at = [&](int q) { return __ffsll((long long)__ballot(mine && ahead == q)) - 1; };
        double sum = 0.0;
        for (int q = 0; q < p.k; ++q) sum += readlane_d(my_s, lane_at(q));
        double cum = 0.0;
        for (int q = 0; q < p.k; ++q) {
            const int l = lane_at(q);
            cum += readlane_d(my_s, l);
            flags |= 1u << l;
            if (cum / sum >= p.tau) break;
        }
    }
    if (mine) mflag[lane] = (uint8_t)((flags >> lane) & 1u);
}

// SplitMix64 output for `state` (Steele, Lea and Flood 2014): golden-gamma
// increment, two xor-shift-multiply rounds, a final xor-shift.
__device__ inline uint64_t splitmix64(uint64_t state) {
    uint64_t z = state + 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

// Phase C for token t: K_final = (K_t ∩ A_trans) refilled from A_trans \ K_t.
template <int EPL>
__device__ void compensate_token(const RouteParams& p, int t, int lane, const int* orig,
                                 const uint8_t* trans, int* fin, double* sbuf, int* n_refill,
                                 int* n_pad) {
    bool in_k[EPL], tr[EPL], take[EPL], fin_f[EPL], out_f[EPL];
    // K_t: lane r < k holds its r-th expert; the list is broadcast lane by lane.
    const int my_orig = lane < p.k ? orig[lane] : -1;
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
        in_k[i] = false;
        tr[i] = lane * EPL + i < p.E && trans[lane * EPL + i];
        take[i] = false;
        out_f[i] = false;
    }
    for (int r = 0; r < p.k; ++r) {
        const int o = __builtin_amdgcn_readlane(my_orig, r);
#pragma unroll
        for (int i = 0; i < EPL; ++i) in_k[i] |= (o == lane * EPL + i);
    }
    const bool kept = my_orig >= 0 && trans[my_orig];
    const uint64_t kept_mask = __ballot(kept);
    const int n_keep = __popcll(kept_mask);
    int avail = 0;   // experts of A_trans outside K_t
#pragma unroll
    for (int i = 0; i < EPL; ++i) avail += __popcll(__ballot(tr[i] && !in_k[i]));
    if (p.refill != CAEE_REFILL_LITERAL && (p.refill == CAEE_REFILL_NONE || n_keep == p.k || avail == 0)) {
        // Nothing to refill: K_final = K_t ∩ A_trans in K_t's own (rank)
        // order.  Each kept slot's score is recomputed by its lane with the
        // same expression as the full pass, and summed in the same order.
        double my_s = 0.0;
        if (kept)
            my_s = p.sslot ? p.sslot[(size_t)t * p.k + lane]
                           : 1.0 / (1.0 + exp(-(double)p.logits[(size_t)t * p.E + my_orig]));
        double total = 0.0;
        for (int r = 0; r < p.k; ++r)
            if ((kept_mask >> r) & 1ull) total += readlane_d(my_s, r);
        const int pos = __popcll(kept_mask & ((1ull << lane) - 1ull));
        if (kept) {
            const size_t o = (size_t)t * p.k + pos;
            fin[pos] = my_orig;
            p.topk_ids[o] = my_orig;
            p.topk_w[o] = (float)(p.rs * (my_s / total));
        }
        if (lane >= n_keep && lane < p.k) {
            const size_t o = (size_t)t * p.k + lane;
            fin[lane] = -1;
            p.topk_ids[o] = -1;
            p.topk_w[o] = 0.0f;
        }
        if (lane == 0 && n_keep < p.k) atomicAdd(n_pad, p.k - n_keep);
        return;
    }
    double s[EPL], key[EPL];
    load_scores<EPL>(p, t, lane, s, key);

    // Refill order: router key (the paper's compensation) or, for the
    // ablation, a 53-bit random key (exact in a double) per (token, expert).
    double rv[EPL];
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
        const uint64_t ctr = ((uint64_t)p.seed << 32) | (uint64_t)(t * p.E + lane * EPL + i);
        rv[i] = p.refill == CAEE_REFILL_RANDOM ? (double)(splitmix64(ctr) >> 11) : key[i];
    }
    // LITERAL: K_final is the top-k of all of A_trans by key (the ordering
    // pass below), no keep-first refill.
    const bool literal = p.refill == CAEE_REFILL_LITERAL;
    const int to_fill = p.refill == CAEE_REFILL_NONE || literal ? 0 : p.k - n_keep;
    int got = 0;
    for (int r = 0; r < to_fill; ++r) {
        double v = -INFINITY;
        int ei = kNoIdx;
#pragma unroll
        for (int i = 0; i < EPL; ++i) {
            if (tr[i] && !in_k[i] && !take[i] && rv[i] > v) {
                v = rv[i];
                ei = lane * EPL + i;
            }
        }
        wave_argmax(v, ei);
        if (ei == kNoIdx) break;
#pragma unroll
        for (int i = 0; i < EPL; ++i)
            if (lane * EPL + i == ei) take[i] = true;
        ++got;
    }
#pragma unroll
    for (int i = 0; i < EPL; ++i) fin_f[i] = literal ? tr[i] : (in_k[i] && tr[i]) || take[i];

    int m = n_keep + got;
    int my_id = -1;   // lane r: the r-th expert of K_final and its score
    double my_s = 0.0;
    if (literal) {
        int n_tr = 0;
#pragma unroll
        for (int i = 0; i < EPL; ++i) n_tr += __popcll(__ballot(tr[i]));
        m = n_tr < p.k ? n_tr : p.k;
    }
    for (int r = 0; r < m; ++r) {
        double v = -INFINITY;
        int ei = kNoIdx;
#pragma unroll
        for (int i = 0; i < EPL; ++i) {
            if (fin_f[i] && !out_f[i] && key[i] > v) {
                v = key[i];
                ei = lane * EPL + i;
            }
        }
        wave_argmax(v, ei);
#pragma unroll
        for (int i = 0; i < EPL; ++i)
            if (lane * EPL + i == ei) out_f[i] = true;
        if (lane == r) my_id = ei;
    }
    my_s = fetch_score<EPL>(s, my_id, lane < m, p.E);
    if (literal) {   // slots that hold an expert from outside K_t
        got = 0;
#pragma unroll
        for (int i = 0; i < EPL; ++i) got += __popcll(__ballot(out_f[i] && !in_k[i]));
    }
    // Weights: scores over their sum in rank order (the same additions on
    // every lane), one slot per lane; slots past m are padding.
    double total = 0.0;
    for (int r = 0; r < m; ++r) total += readlane_d(my_s, r);
    if (lane < p.k) {
        const size_t o = (size_t)t * p.k + lane;
        const bool have = lane < m;
        fin[lane] = have ? my_id : -1;
        p.topk_ids[o] = have ? my_id : -1;
        p.topk_w[o] = have ? (float)(p.rs * (my_s / total)) : 0.0f;
    }
    if (lane == 0) {
        atomicAdd(n_refill, got);
        atomicAdd(n_pad, p.k - m);
    }
}

// Routing kernel: one wavefront per token (phase A).  Block 0 also resets
// the counters the later kernels of this call accumulate into.
template <int EPL>
__global__ __launch_bounds__(kTokThreads) void k_route_tokens(RouteParams p) {
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int t = blockIdx.x * kTokWaves + wave;
    if (blockIdx.x == 0 && threadIdx.x < 4) p.counters[threadIdx.x] = 0;
    if (t < p.T)
        route_token<EPL>(p, t, lane, p.orig_ids + (size_t)t * p.k, p.gbuf + (size_t)t * p.k, p.top1 + t,
                         p.mflag + (size_t)t * p.k);
}

// Batch-summed importance (SUM rule): one wavefront per expert adds the
// expert's gate weights in ascending token order.
__device__ void importance_sum_expert(const RouteParams& p, int e, int lane) {
    double sum = 0.0;
    for (int t0 = 0; t0 < p.T; t0 += kWave) {
        const int t = t0 + lane;
        double v = 0.0;
        bool hit = false;
        if (t < p.T) {
            for (int r = 0; r < p.k; ++r) {
                if (p.orig_ids[(size_t)t * p.k + r] == e) {
                    v = p.gbuf[(size_t)t * p.k + r];
                    hit = true;
                }
            }
        }
        unsigned long long m = __ballot(hit);
        while (m) {
            const int l = __ffsll((long long)m) - 1;
            sum += readlane_d(v, l);
            m &= m - 1;
        }
    }
    if (lane == 0) p.imp_sum[e] = sum;
}

// The same sums for small batches, one thread per expert walking the
// (token, slot) pairs in order (reads of one LDS word by every thread).
__device__ void importance_sum_small(const RouteParams& p, int tid, int nthr) {
    const int n = p.T * p.k;
    for (int e = tid; e < p.E; e += nthr) {
        double sum = 0.0;
        for (int i = 0; i < n; ++i)
            if (p.orig_ids[i] == e) sum += p.gbuf[i];
        p.imp_sum[e] = sum;
    }
}

__global__ __launch_bounds__(kTokThreads) void k_importance_sum(RouteParams p) {
    const int e = blockIdx.x * kTokWaves + threadIdx.x / kWave;
    if (e < p.E) importance_sum_expert(p, e, threadIdx.x & (kWave - 1));
}

// Pruning kernel (one workgroup): Sec. IV-B steps 1-4 over the whole batch.
// Bin loads are float64 sums of fp32 costs; while a bin's nonzero costs span
// less than 2^20 every such sum is exact, so the order of the additions (LDS
// atomics here) does not change any value or decision.
struct PruneShared {
    unsigned long long imp[kMaxE];
    uint8_t act[kMaxE], must[kMaxE], prom[kMaxE];
    float cost[kMaxE];
    int bin[kMaxE];
    int cand[kMaxE];        // candidates as gathered
    unsigned long long cimp[kMaxE];   // their importance bits
    int sorted[kMaxE];      // candidates in visiting order
    int cbin[kMaxE];        // their bins
    float ccost[kMaxE];     // their costs
    double aload[kMaxBins], mload[kMaxBins];
    double fbase;
    int ncand;
    int stat[5];            // step-4 counts: active, mandatory, promoted, pruned, kept
    int fallback;           // A_trans came out empty: steps 2-3 rerun with each token's top expert mandatory
};

// Steps 2-3 of Sec. IV-B from the membership in sh.act / sh.must: per-bin
// loads of A_act and A_must, F_base, the candidates (active, not mandatory)
// in visiting order (importance descending, index ascending), and the
// cost-invariant expansion into sh.prom, one bin per thread (bins are
// independent).  Expects sh.prom, the loads and the candidate count zeroed.
// Ends with a barrier.
__device__ void prune_expand(const RouteParams& p, int tid, int nthr, PruneShared& sh) {
    const int lane = tid & (kWave - 1);
    const int wave = tid / kWave;
    const int E = p.E, nb = p.n_bins;
    for (int e = tid; e < E; e += nthr) {
        const double c = (double)sh.cost[e];
        const int b = sh.bin[e];
        if (sh.act[e] && b >= 0) atomicAdd(&sh.aload[b], c);
        if (sh.must[e] && b >= 0) atomicAdd(&sh.mload[b], c);
        if (sh.act[e] && !sh.must[e]) {
            const int i = atomicAdd(&sh.ncand, 1);
            sh.cand[i] = e;
            sh.cimp[i] = sh.imp[e];
        }
    }
    __syncthreads();
    const int n_cand = sh.ncand;
    for (int i = tid; i < n_cand; i += nthr) {
        const int e = sh.cand[i];
        const unsigned long long ie = sh.cimp[i];
        int rank = 0;
        for (int j = 0; j < n_cand; ++j) {
            const unsigned long long io = sh.cimp[j];
            const int o = sh.cand[j];
            rank += (io > ie || (io == ie && o < e)) ? 1 : 0;
        }
        sh.sorted[rank] = e;
        sh.cbin[rank] = sh.bin[e];
        sh.ccost[rank] = sh.cost[e];
    }
    __syncthreads();
    if (wave == 0) {
        double fb = 0.0;
        for (int b = lane; b < nb; b += kWave) fb = fmax(fb, sh.mload[b]);
        fb = wave_max_d(fb);
        if (lane == 0) sh.fbase = fb;
    }
    for (int b = tid; b < nb && p.bin_loads; b += nthr) {
        p.bin_loads[b] = sh.aload[b];
        p.bin_loads[nb + b] = sh.mload[b];
    }
    __syncthreads();

    // Step 3: expansion, walking the candidates in visiting order.
    const double fbase = sh.fbase;
    for (int b = tid; b < nb; b += nthr) {
        double load = sh.mload[b];
        for (int r = 0; r < n_cand; ++r) {
            if (sh.cbin[r] != b) continue;
            const double c = (double)sh.ccost[r];
            if (load + c <= fbase) {
                sh.prom[sh.sorted[r]] = 1;
                load += c;
            }
        }
        if (p.bin_loads) p.bin_loads[2 * nb + b] = load;
    }
    __syncthreads();
}

// Run by one workgroup of `nthr` threads (a multiple of the wave size).
__device__ void prune_all(const RouteParams& p, int tid, int nthr, PruneShared& sh) {
    unsigned long long* s_imp = sh.imp;
    uint8_t *s_act = sh.act, *s_must = sh.must, *s_prom = sh.prom;
    float* s_cost = sh.cost;
    int* s_bin = sh.bin;
    double *s_aload = sh.aload, *s_mload = sh.mload;
    int& s_ncand = sh.ncand;
    const int lane = tid & (kWave - 1);
    const int wave = tid / kWave;
    const int T = p.T, E = p.E, k = p.k, nb = p.n_bins;

    for (int e = tid; e < E; e += nthr) {
        s_imp[e] = 0ull;
        s_act[e] = s_must[e] = s_prom[e] = 0;
        s_cost[e] = p.cost[e];
        const int b = p.bin ? p.bin[e] : 0;
        s_bin[e] = (b >= 0 && b < nb) ? b : -1;   // out-of-range bins (a precondition violation) count nowhere
    }
    for (int b = tid; b < nb; b += nthr) s_aload[b] = s_mload[b] = 0.0;
    if (tid == 0) {
        s_ncand = 0;
        sh.fallback = 0;
    }
    if (tid < 5) sh.stat[tid] = 0;
    __syncthreads();

    // Step 1: A_act, importance, A_must (pairs mandatory on their own, and
    // for the SUM rule every expert whose summed weight reaches tau).
    // Batches of 8 pairs per thread: their loads are issued together.
    constexpr int kB = 8;
    for (int i0 = tid; i0 < T * k; i0 += kB * nthr) {
        int ev[kB];
        double gv[kB];
        uint8_t mv[kB];
#pragma unroll
        for (int b = 0; b < kB; ++b) {
            const int i = i0 + b * nthr;
            const bool in = i < T * k;
            ev[b] = in ? p.orig_ids[i] : -1;
            gv[b] = in ? p.gbuf[i] : 0.0;
            mv[b] = in ? p.mflag[i] : 0;
        }
#pragma unroll
        for (int b = 0; b < kB; ++b) {
            if (ev[b] < 0) continue;
            atomicMax(&s_imp[ev[b]], (unsigned long long)__double_as_longlong(gv[b]));
            s_act[ev[b]] = 1;
            if (mv[b]) s_must[ev[b]] = 1;
        }
    }
    __syncthreads();
    if (p.rule == CAEE_IMPORTANCE_SUM) {
        for (int e = tid; e < E; e += nthr) {
            if (!s_act[e]) continue;
            const double I = p.imp_sum[e];
            s_imp[e] = (unsigned long long)__double_as_longlong(I);
            if (I >= p.tau) s_must[e] = 1;
        }
        __syncthreads();
    }

    prune_expand(p, tid, nthr, sh);
    // A_trans = A_must + promoted is empty only when no thread sees a member.
    // Then Sec. IV-C's final top-k would have nothing to choose from: steps
    // 2-3 run again with every token's own top expert mandatory (the only
    // departure from step 1 as written).
    bool member = false;
    for (int e = tid; e < E; e += nthr) member |= (s_must[e] | s_prom[e]) != 0;
    if (!__syncthreads_or(member)) {   // (nothing was promoted either: s_prom stays zero)
        for (int t = tid; t < T; t += nthr) s_must[p.top1[t]] = 1;
        for (int b = tid; b < nb; b += nthr) s_aload[b] = s_mload[b] = 0.0;
        if (tid == 0) {
            s_ncand = 0;
            sh.fallback = 1;
        }
        __syncthreads();
        prune_expand(p, tid, nthr, sh);
    }
    const int n_cand = s_ncand;

    // Step 4: A_trans = A_must + promoted; masks and counters by ballot,
    // one 64-expert block per wave, counts added in LDS.
    for (int e = tid; e < E; e += nthr) p.trans[e] = s_must[e] | s_prom[e];
    const int words = (E + 31) / 32;
    for (int base = wave * kWave; base < E; base += nthr) {
        const int e = base + lane;
        const bool v = e < E;
        const bool act = v && s_act[e], must = v && s_must[e], prom = v && s_prom[e];
        const bool trans = must || prom;
        const unsigned long long ba = __ballot(act), bm = __ballot(must), bt = __ballot(trans),
                                 bp = __ballot(act && !trans), bpr = __ballot(prom);
        if (lane == 0) {
            atomicAdd(&sh.stat[0], __popcll(ba));
            atomicAdd(&sh.stat[1], __popcll(bm));
            atomicAdd(&sh.stat[2], __popcll(bpr));
            atomicAdd(&sh.stat[3], __popcll(bp));
            atomicAdd(&sh.stat[4], __popcll(bt));
        }
        if (p.masks && lane < 2) {
            const int w = base / 32 + lane;
            if (w < words) {
                const int sh_ = 32 * lane;
                p.masks[w] = (uint32_t)(ba >> sh_);
                p.masks[words + w] = (uint32_t)(bm >> sh_);
                p.masks[2 * words + w] = (uint32_t)(bt >> sh_);
                p.masks[3 * words + w] = (uint32_t)(bp >> sh_);
            }
        }
    }
    __syncthreads();
    if (p.stats && tid == 0) {
        p.stats[0] = sh.stat[0];   // |A_act|
        p.stats[1] = sh.stat[1];   // |A_must|
        p.stats[2] = n_cand;
        p.stats[3] = sh.stat[2];   // promoted
        p.stats[4] = sh.stat[3];   // pruned
        p.stats[5] = sh.stat[4];   // |A_trans|
        p.stats[8] = sh.fallback;
    }
}

__global__ __launch_bounds__(kRouteThreads) void k_prune(RouteParams p) {
    __shared__ PruneShared sh;
    prune_all(p, threadIdx.x, kRouteThreads, sh);
}

// Row offsets of every expert slot and the FFN work lists, from the slot
// row counts in s_cnt (run by one wavefront).  Slot x (x < E routed, E+s
// shared) owns rows [off[x], off[x] + count); the shared slots come first
// (shared expert s owns rows s*T .. s*T + T - 1, known before routing), then
// the routed ones in expert order.  Then one small chunk per slot with at
// most chunk_small rows, and ceil(rows / chunk_big) near-equal big chunks per
// larger slot, the small chunks listed first.
__device__ void build_lists(const RouteParams& p, const int* s_cnt, int* s_off, int tid) {
    // Run by the first four waves of the workgroup (every thread calls it:
    // it holds a barrier).  Lane gl of the 256 takes slots [gl*per, gl*per+per)
    // in row order, so the scans below follow the slots' row order.
    constexpr int kW = 4;
    __shared__ int s_tot[kW][3];
    const int nx = p.E + p.n_shared, ns = p.n_shared, E = p.E;
    const int cs = p.chunk_small, cb = p.chunk_big;
    const int lane = tid & (kWave - 1), wave = tid / kWave;
    const bool active = wave < kW;   // uniform per wave
    const int per = (nx + kW * kWave - 1) / (kW * kWave);
    const int gl = wave * kWave + lane;
    const int lo = gl * per;
    const int hi = min(lo + per, nx);
    auto slot_at = [&](int j) { return j < ns ? E + j : j - ns; };   // j-th slot in row order
    int sum = 0, ssum = 0, bsum = 0, inc = 0, sinc = 0, binc = 0;
    if (active) {
        for (int j = lo; j < hi; ++j) {
            const int n = s_cnt[slot_at(j)];
            sum += n;
            ssum += (n > 0 && n <= cs) ? 1 : 0;
            bsum += n > cs ? (n + cb - 1) / cb : 0;
        }
        inc = wave_incl_scan(sum);
        sinc = wave_incl_scan(ssum);
        binc = wave_incl_scan(bsum);
        if (lane == kWave - 1) {
            s_tot[wave][0] = inc;
            s_tot[wave][1] = sinc;
            s_tot[wave][2] = binc;
        }
    }
    __syncthreads();
    if (!active) return;
    int base = 0, sbase = 0, bbase = 0, total = 0, stotal = 0, btotal = 0;
    for (int w = 0; w < kW; ++w) {
        if (w < wave) {
            base += s_tot[w][0];
            sbase += s_tot[w][1];
            bbase += s_tot[w][2];
        }
        total += s_tot[w][0];
        stotal += s_tot[w][1];
        btotal += s_tot[w][2];
    }
    int run = base + inc - sum, srun = sbase + sinc - ssum, brun = stotal + bbase + binc - bsum;
    for (int j = lo; j < hi; ++j) {
        const int x = slot_at(j);
        const int cnt = s_cnt[x];
        s_off[x] = run;
        p.perm_off[x] = run;
        if (cnt > 0 && cnt <= cs) {
            int* chk = p.chunks + 4 * srun++;
            chk[0] = x;
            chk[1] = run;
            chk[2] = cnt;
            chk[3] = 0;
        } else if (cnt > cs) {
            const int pieces = (cnt + cb - 1) / cb;
            const int size = (cnt + pieces - 1) / pieces;
            for (int c = 0; c < pieces; ++c) {
                int* chk = p.chunks + 4 * (brun + c);
                chk[0] = x;
                chk[1] = run + c * size;
                chk[2] = min(size, cnt - c * size);
                // Pieces 2i and 2i + 1 form a pair (rows adjacent, at most
                // 2 * chunk_big together); a last odd piece has none.
                chk[3] = (c & 1) ? -1 : (c + 1 < pieces ? 1 : 0);
            }
            brun += pieces;
        }
        run += cnt;
    }
    if (gl == 0) {
        s_off[nx] = total;
        p.perm_off[nx] = total;
        p.n_chunks[0] = stotal;
        p.n_chunks[1] = btotal;
    }
}

// Token-block bitmasks: bit (t - t0) of word (x, (t - t0) / 64) is set when
// token t of [t0, t0 + tn) chose routed expert x.  W words per expert.  An
// expert named twice in one token's list sets one bit: it gets one row, which
// both slots read.
__device__ void token_masks(const RouteParams& p, int t0, int tn, int W, int tid, int nthr,
                            unsigned long long* s_mask) {
    const int E = p.E, k = p.k;
    for (int i = tid; i < E * W; i += nthr) s_mask[i] = 0ull;
    __syncthreads();
    for (int i = tid; i < tn * k; i += nthr) {
        const int e = p.topk_ids[(size_t)t0 * k + i];
        if (e >= 0 && e < E) {
            const int tl = i / k;
            atomicOr(&s_mask[e * W + (tl >> 6)], 1ull << (tl & 63));
        }
    }
    __syncthreads();
}

// The bitmasks, and per word the number of set bits in the words before it.
__device__ void fill_masks(const RouteParams& p, int t0, int tn, int W, int tid, int nthr,
                           unsigned long long* s_mask, int* s_pre) {
    const int E = p.E;
    token_masks(p, t0, tn, W, tid, nthr, s_mask);
    // s_pre[e*W + w]: tokens of words 0..w-1 that chose expert e.
    for (int i = tid; i < E * W; i += nthr) {
        const int w = i % W;
        int c = 0;
        for (int v = i - w; v < i; ++v) c += __popcll(s_mask[v]);
        s_pre[i] = c;
    }
    __syncthreads();
}

// Rows of the (token, slot) entries of tokens [t0, t0 + tn): routed entry
// of expert e goes to row base[e] + (number of earlier tokens of the block
// that chose e); caller-supplied ids outside [0, E) are empty slots.
__device__ void place_entries(const RouteParams& p, int t0, int tn, int W, const int* base, int tid, int nthr,
                              const unsigned long long* s_mask, const int* s_pre) {
    const int E = p.E, k = p.k, slots = k + p.n_shared;
    for (int i = tid; i < tn * k; i += nthr) {
        const int tl = i / k, j = i - tl * k;
        const int t = t0 + tl;
        const int e = p.topk_ids[(size_t)t * k + j];
        if (e < 0 || e >= E) {
            p.perm_pos[(size_t)t * slots + j] = -1;
            continue;
        }
        const int w = e * W + (tl >> 6);
        const int rank = s_pre[w] + __popcll(s_mask[w] & ((1ull << (tl & 63)) - 1ull));
        const int pos = base[e] + rank;
        p.perm_tok[pos] = t;
        p.perm_pos[(size_t)t * slots + j] = pos;
    }
}

// Shared experts: every token, in order.
__device__ void place_shared(const RouteParams& p, const int* s_off, int tid, int nthr) {
    const int T = p.T, E = p.E, k = p.k, slots = k + p.n_shared;
    for (int i = tid; i < T * p.n_shared; i += nthr) {
        const int t = i / p.n_shared, sh = i - t * p.n_shared;
        const int pos = s_off[E + sh] + t;
        p.perm_tok[pos] = t;
        p.perm_pos[(size_t)t * slots + k + sh] = pos;
    }
}

// Permutation of K_final (read from global memory) by expert slot, tokens
// ascending within a slot, plus the FFN work lists, for batches of at most
// kMaskT tokens: one workgroup; each expert's tokens are a bitmask in LDS and
// every (token, slot) entry finds its row independently by counting set bits.
// Also reports the refill/empty-slot counts of the compensation kernel.
struct PermShared {
    int cnt[kMaxE + kMaxShared];
    int off[kMaxE + kMaxShared + 1];
    unsigned long long mask[kMaxE * (kMaskT / 64)];
    int pre[kMaxE * (kMaskT / 64)];
};

__device__ void permute_small(const RouteParams& p, int tid, int nthr, PermShared& sh) {
    int* s_cnt = sh.cnt;
    int* s_off = sh.off;
    unsigned long long* s_mask = sh.mask;
    if (tid == 0 && p.stats) {
        p.stats[6] = p.counters[1];
        p.stats[7] = p.counters[2];
    }
    if (!p.do_permute) return;
    const int T = p.T, E = p.E;
    const int W = (T + 63) / 64;
    fill_masks(p, 0, T, W, tid, nthr, s_mask, sh.pre);
    for (int x = tid; x < E + p.n_shared; x += nthr) {
        int c = T;
        if (x < E) {
            c = 0;
            for (int w = 0; w < W; ++w) c += __popcll(s_mask[x * W + w]);
        }
        s_cnt[x] = c;
    }
    __syncthreads();
    build_lists(p, s_cnt, s_off, tid);
    __syncthreads();
    place_shared(p, s_off, tid, nthr);
    place_entries(p, 0, T, W, s_off, tid, nthr, s_mask, sh.pre);
}

__global__ __launch_bounds__(kRouteThreads) void k_permute(RouteParams p) {
    __shared__ PermShared sh;
    permute_small(p, threadIdx.x, kRouteThreads, sh);
}

// Larger batches: the tokens are cut into blocks of kMaskT.
// (1) per block, each routed expert's token count;
// counted from the same bitmasks (k_permute_place) as the rows are placed,
// so a repeated expert in one token's list counts once;
__global__ __launch_bounds__(kRouteThreads) void k_permute_count(RouteParams p) {
    __shared__ unsigned long long s_mask[kMaxE * (kMaskT / 64)];
    const int tid = threadIdx.x, b = blockIdx.x;
    const int t0 = b * kMaskT, tn = min(kMaskT, p.T - t0);
    const int W = (tn + 63) / 64;
    token_masks(p, t0, tn, W, tid, kRouteThreads, s_mask);
    for (int e = tid; e < p.E; e += kRouteThreads) {
        int c = 0;
        for (int w = 0; w < W; ++w) c += __popcll(s_mask[e * W + w]);
        p.perm_blk[(size_t)b * p.E + e] = c;
    }
}

// (2) one workgroup: slot totals, offsets and work lists, each block's first
// row per expert (replacing its count), the shared experts' rows;
__global__ __launch_bounds__(kRouteThreads) void k_permute_scan(RouteParams p) {
    __shared__ int s_cnt[kMaxE + kMaxShared];
    __shared__ int s_off[kMaxE + kMaxShared + 1];
    const int tid = threadIdx.x, E = p.E;
    const int nblk = (p.T + kMaskT - 1) / kMaskT;
    if (tid == 0 && p.stats) {
        p.stats[6] = p.counters[1];
        p.stats[7] = p.counters[2];
    }
    for (int x = tid; x < E + p.n_shared; x += kRouteThreads) {
        int c = p.T;
        if (x < E) {
            c = 0;
            for (int b = 0; b < nblk; ++b) c += p.perm_blk[(size_t)b * E + x];
        }
        s_cnt[x] = c;
    }
    __syncthreads();
    build_lists(p, s_cnt, s_off, tid);
    __syncthreads();
    for (int x = tid; x < E; x += kRouteThreads) {
        int run = s_off[x];
        for (int b = 0; b < nblk; ++b) {
            const int c = p.perm_blk[(size_t)b * E + x];
            p.perm_blk[(size_t)b * E + x] = run;
            run += c;
        }
    }
    place_shared(p, s_off, tid, kRouteThreads);
}

// (3) per block, the rows of its (token, slot) entries.
__global__ __launch_bounds__(kRouteThreads) void k_permute_place(RouteParams p) {
    __shared__ unsigned long long s_mask[kMaxE * (kMaskT / 64)];
    __shared__ int s_pre[kMaxE * (kMaskT / 64)];
    const int tid = threadIdx.x, b = blockIdx.x;
    const int t0 = b * kMaskT, tn = min(kMaskT, p.T - t0);
    const int W = (tn + 63) / 64;
    fill_masks(p, t0, tn, W, tid, kRouteThreads, s_mask, s_pre);
    place_entries(p, t0, tn, W, p.perm_blk + (size_t)b * p.E, tid, kRouteThreads, s_mask, s_pre);
}

hipError_t launch_permutation(const RouteParams& p, hipStream_t s) {
    if (!p.do_permute || p.T <= kMaskT) {
        hipLaunchKernelGGL(k_permute, dim3(1), dim3(kRouteThreads), 0, s, p);
        return hipGetLastError();
    }
    const dim3 blocks((p.T + kMaskT - 1) / kMaskT);
    hipLaunchKernelGGL(k_permute_count, blocks, dim3(kRouteThreads), 0, s, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_permute_scan, dim3(1), dim3(kRouteThreads), 0, s, p);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_permute_place, blocks, dim3(kRouteThreads), 0, s, p);
    return hipGetLastError();
}

// Compensation kernel: one wavefront per token (phase C).
template <int EPL>
__global__ __launch_bounds__(kTokThreads) void k_compensate(RouteParams p) {
    __shared__ uint8_t s_trans[kMaxE];
    __shared__ double s_sbuf[kTokWaves][kMaxK];
    __shared__ int s_fin[kTokWaves][kMaxK];
    __shared__ int s_cnt[2];   // refilled and empty slots of the workgroup's tokens
    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wave = tid / kWave;
    for (int e = tid; e < p.E; e += kTokThreads) s_trans[e] = p.trans[e];
    if (tid < 2) s_cnt[tid] = 0;
    __syncthreads();
    for (int t = blockIdx.x * kTokWaves + wave; t < p.T; t += gridDim.x * kTokWaves)
        compensate_token<EPL>(p, t, lane, p.orig_ids + (size_t)t * p.k, s_trans, s_fin[wave], s_sbuf[wave],
                              &s_cnt[0], &s_cnt[1]);
    // One global update per workgroup (per-token updates of the same two
    // words serialise in the L2).
    __syncthreads();
    if (tid == 0) {
        if (s_cnt[0]) atomicAdd(&p.counters[1], s_cnt[0]);
        if (s_cnt[1]) atomicAdd(&p.counters[2], s_cnt[1]);
    }
}

// Small batches: the whole routing step (phases A-C and the permutation)
// in one workgroup of 16 wavefronts, one launch instead of four or five.
// Phases are separated by workgroup barriers.  Everything one phase hands to
// the next (K_t, G, the mandatory flags, the cost and bin tables, A_trans,
// K_final and its weights, the counters) stays in LDS: the phases run on a
// copy of the parameters whose arrays point there, and the results the
// caller and the FFN read are copied out at the end.
constexpr int kFusedWaves = kRouteThreads / kWave;

template <int EPL>
__device__ void route_fused_body(const RouteParams& p) {
    __shared__ double s_sbuf[kFusedWaves][kMaxK];
    __shared__ int s_ids[kFusedWaves][kMaxK];
    __shared__ PruneShared sp;
    __shared__ PermShared sq;
    __shared__ int32_t l_orig[kFusedT * kMaxK], l_top1[kFusedT], l_fin[kFusedT * kMaxK], l_ctr[4];
    __shared__ double l_g[kFusedT * kMaxK], l_isum[kMaxE];
    __shared__ float l_w[kFusedT * kMaxK], l_cost[kMaxE];
    __shared__ int32_t l_bin[kMaxE];
    __shared__ uint8_t l_mflag[kFusedT * kMaxK], l_trans[kMaxE];
    __shared__ uint32_t l_masks[4 * (kMaxE / 32)];
    __shared__ int32_t l_stats[kStats];
    __shared__ double l_bl[3 * kMaxE];
    __shared__ double l_s[kFusedT * kMaxK];
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    const int k = p.k, E = p.E;
    RouteParams q = p;
    q.orig_ids = l_orig;
    q.gbuf = l_g;
    q.top1 = l_top1;
    q.mflag = l_mflag;
    q.cost = l_cost;
    q.bin = p.bin ? l_bin : nullptr;
    q.trans = l_trans;
    q.topk_ids = l_fin;
    q.topk_w = l_w;
    q.counters = l_ctr;
    q.imp_sum = l_isum;
    q.masks = p.masks ? l_masks : nullptr;
    q.stats = p.stats ? l_stats : nullptr;
    q.bin_loads = p.bin_loads && p.n_bins <= kMaxE ? l_bl : p.bin_loads;
    q.sslot = l_s;
    // The tables, read by the waves that route no token while the others do.
    for (int e = tid; e < E; e += kRouteThreads) {
        l_cost[e] = p.cost[e];
        if (p.bin) l_bin[e] = p.bin[e];
    }
    if (tid < 4) l_ctr[tid] = 0;
    for (int t = wave; t < p.T; t += kFusedWaves)
        route_token<EPL>(q, t, lane, q.orig_ids + (size_t)t * k, q.gbuf + (size_t)t * k, q.top1 + t,
                         q.mflag + (size_t)t * k);
    __syncthreads();
    if (p.rule == CAEE_IMPORTANCE_SUM) {
        importance_sum_small(q, tid, kRouteThreads);
        __syncthreads();
    }
    prune_all(q, tid, kRouteThreads, sp);
    __syncthreads();
    __shared__ int s_cnt[2];
    if (tid < 2) s_cnt[tid] = 0;
    __syncthreads();
    for (int t = wave; t < p.T; t += kFusedWaves)
        compensate_token<EPL>(q, t, lane, q.orig_ids + (size_t)t * k, l_trans, s_ids[wave], s_sbuf[wave],
                              &s_cnt[0], &s_cnt[1]);
    __syncthreads();
    if (tid == 0) {   // the only workgroup: the call's totals
        l_ctr[1] = s_cnt[0];
        l_ctr[2] = s_cnt[1];
    }
    __syncthreads();
    if (p.do_permute || p.stats) permute_small(q, tid, kRouteThreads, sq);
    // Results read after this kernel: K_t, K_final and its weights, A_trans.
    for (int i = tid; i < p.T * k; i += kRouteThreads) {
        p.orig_ids[i] = l_orig[i];
        p.topk_ids[i] = l_fin[i];
        p.topk_w[i] = l_w[i];
    }
    for (int e = tid; e < E; e += kRouteThreads) p.trans[e] = l_trans[e];
    if (tid < 4) p.counters[tid] = l_ctr[tid];
    const int words = (E + 31) / 32;
    if (p.masks)
        for (int i = tid; i < 4 * words; i += kRouteThreads) p.masks[i] = l_masks[i];
    if (p.stats && tid < kStats) p.stats[tid] = l_stats[tid];
    if (q.bin_loads == l_bl)
        for (int i = tid; i < 3 * p.n_bins; i += kRouteThreads) p.bin_loads[i] = l_bl[i];
}

template <int EPL>
__global__ __launch_bounds__(kRouteThreads) void k_route_fused(RouteParams p) {
    route_fused_body<EPL>(p);
}

// The shared experts' gate/up for a batch of at most 16 tokens, run by the
// workgroups after the first in the routing launch.  Item = one 16-column
// tile (gate and up rows) of one shared expert; the 16 waves of the
// workgroup take consecutive ranges of the contraction, and wave 0 adds the
// 16 partial sums in wave order (deterministic) and stores the SwiGLU rows.
// Shared expert s owns rows s*T .. s*T + T - 1 (row s*T + t for token t).
template <class M>
__device__ void shared_gate_up(const FfnParams& p, int wg, int n_wg) {
    constexpr int kWaves = kRouteThreads / kWave;
    __shared__ f32x4_t s_part[kWaves][2][kWave];
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int r = lane & 15, g = lane >> 4;
    const int tiles = p.f / 16;
    const size_t row_units = (size_t)p.d * M::kElemBytes / 16;
    const int ksteps = (int)(row_units / 4);
    const int kper = (ksteps + kWaves - 1) / kWaves;
    const int k0 = min(ksteps, wave * kper), k1 = min(ksteps, k0 + kper);
    const size_t expert_bytes = (size_t)2 * p.f * p.d * M::kElemBytes;
    const int astep = p.tiled ? 64 : 4;
    for (int item = wg; item < p.n_shared * tiles; item += n_wg) {
        const int sh = item / tiles, jt = item - sh * tiles;
        const u32x4_t* wb = (const u32x4_t*)((const char*)p.sh_w13 + (size_t)sh * expert_bytes);
        const u32x4_t* const a[2] = {
            p.tiled ? wb + ((size_t)jt * ksteps + k0) * 64 + lane
                    : wb + (size_t)(jt * 16 + r) * row_units + g + 4 * (size_t)k0,
            p.tiled ? wb + ((size_t)(tiles + jt) * ksteps + k0) * 64 + lane
                    : wb + (size_t)(p.f + jt * 16 + r) * row_units + g + 4 * (size_t)k0};
        const int t = r < p.T ? r : 0;   // padded token columns read a valid row; results dropped
        const u32x4_t* const xb[1] = {(const u32x4_t*)p.x + (size_t)t * row_units + g + 4 * (size_t)k0};
        f32x4_t acc[2][1] = {{f32x4_t{0.f, 0.f, 0.f, 0.f}}, {f32x4_t{0.f, 0.f, 0.f, 0.f}}};
        if (k1 > k0) tile_contract<M, kRouteSharedU, 2, 1>(a, astep, xb, 1, k1 - k0, acc);   // short rows leave waves idle
        s_part[wave][0][lane] = acc[0][0];
        s_part[wave][1][lane] = acc[1][0];
        __syncthreads();
        if (wave == 0 && r < p.T) {
            f32x4_t gs = s_part[0][0][lane], us = s_part[0][1][lane];
            for (int w = 1; w < kWaves; ++w) {
                gs += s_part[w][0][lane];
                us += s_part[w][1][lane];
            }
            float h[4];
#pragma unroll
            for (int v = 0; v < 4; ++v) h[v] = silu_mul(gs[v], us[v]);
            store_h<M>(p, (size_t)(sh * p.T + r) * p.f + jt * 16 + 4 * g, h);
        }
        __syncthreads();
    }
}

template <int EPL, class M>
__global__ __launch_bounds__(kRouteThreads) void k_route_fused_shared(RouteParams p, FfnParams fp) {
    if (blockIdx.x == 0) route_fused_body<EPL>(p);
    else shared_gate_up<M>(fp, blockIdx.x - 1, gridDim.x - 1);
}

}  // namespace

bool route_runs_shared(const caee_layer_desc_t& d) {
    // one 16-token block: the workgroups' tiles hold every token of the batch
    return kRouteShared && d.T <= 16 && d.T <= kFusedT && d.n_shared > 0 && d.w_dtype != CAEE_FP8_E4M3;
}

hipError_t launch_route_shared(const RouteParams& p, const FfnParams& fp, int w_dtype, hipStream_t s) {
    const int items = fp.n_shared * (fp.f / 16);
    const int cap = device_cu_count() - 1;
    const dim3 grid(1 + (items < cap ? items : cap));
    auto go = [&](auto k) -> hipError_t {
        hipLaunchKernelGGL(k, grid, dim3(kRouteThreads), 0, s, p, fp);
        return hipGetLastError();
    };
    const bool bf16 = w_dtype == CAEE_BF16;
    if (w_dtype != CAEE_BF16 && w_dtype != CAEE_F32) return hipErrorInvalidValue;
    switch (p.epl) {
        case 1: return bf16 ? go(k_route_fused_shared<1, Bf16Math>) : go(k_route_fused_shared<1, F32Math>);
        case 2: return bf16 ? go(k_route_fused_shared<2, Bf16Math>) : go(k_route_fused_shared<2, F32Math>);
        case 4: return bf16 ? go(k_route_fused_shared<4, Bf16Math>) : go(k_route_fused_shared<4, F32Math>);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_route(const RouteParams& p, hipStream_t s) {
    const dim3 tok_grid((p.T + kTokWaves - 1) / kTokWaves);
    auto token_kernels = [&](auto route_k, auto comp_k, auto fused_k) -> hipError_t {
        if (p.T <= kFusedT) {
            hipLaunchKernelGGL(fused_k, dim3(1), dim3(kRouteThreads), 0, s, p);
            return hipGetLastError();
        }
        hipLaunchKernelGGL(route_k, tok_grid, dim3(kTokThreads), 0, s, p);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        if (p.rule == CAEE_IMPORTANCE_SUM) {
            hipLaunchKernelGGL(k_importance_sum, dim3((p.E + kTokWaves - 1) / kTokWaves), dim3(kTokThreads), 0, s, p);
            e = hipGetLastError();
            if (e != hipSuccess) return e;
        }
        hipLaunchKernelGGL(k_prune, dim3(1), dim3(kRouteThreads), 0, s, p);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(comp_k, tok_grid, dim3(kTokThreads), 0, s, p);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        if (!p.do_permute && !p.stats) return hipSuccess;
        return launch_permutation(p, s);
    };
    switch (p.epl) {
        case 1: return token_kernels(k_route_tokens<1>, k_compensate<1>, k_route_fused<1>);
        case 2: return token_kernels(k_route_tokens<2>, k_compensate<2>, k_route_fused<2>);
        case 4: return token_kernels(k_route_tokens<4>, k_compensate<4>, k_route_fused<4>);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_permute(const RouteParams& p, hipStream_t s) {
    RouteParams q = p;
    q.stats = nullptr;   // counters are not filled when routing did not run
    return launch_permutation(q, s);
}

}  // namespace caee
