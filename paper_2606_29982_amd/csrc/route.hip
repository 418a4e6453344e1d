// Routing, cost-aware pruning, compensation and token permutation for one
// MoE layer call, in a single 1024-thread workgroup (decode batches).
//
//   phase A (one wavefront per token): sigmoid scores, group-limited top-k
//            K_t and normalised gate weights G(t)_e (Sec. II-A);
//   phase B (whole workgroup): importance, mandatory/candidate split,
//            per-bin baseline cost F_base and cost-invariant expansion
//            (Sec. IV-A, IV-B steps 1-4);
//   phase C (one wavefront per token): masking of pruned experts and
//            top-k refill from A_trans (Sec. IV-C), weight renormalisation;
//   permute: stable counting sort of the (token, expert) pairs by expert,
//            shared experts last, and the FFN work list (expert chunks of
//            at most kChunkTokens rows).
//
// Every decision is taken in float64 with ties to the lower index, so the
// result does not depend on the order in which lanes or waves finish.
#include <math.h>

#include "caee_internal.h"

namespace caee {
namespace {

constexpr int kRouteWaves = kRouteThreads / kWave;
constexpr int kNoIdx = 0x7fffffff;

// Larger value wins; equal values go to the lower index.
__device__ inline void argmax_merge(double& v, int& i, double ov, int oi) {
    if (ov > v || (ov == v && oi < i)) {
        v = ov;
        i = oi;
    }
}

__device__ inline void wave_argmax(double& v, int& i) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        const double ov = __shfl_xor(v, off);
        const int oi = __shfl_xor(i, off);
        argmax_merge(v, i, ov, oi);
    }
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

// Broadcast s of expert `e` from the lane that holds it.
template <int EPL>
__device__ inline double score_of(const double (&s)[EPL], int lane, int e) {
    double mine = 0.0;
#pragma unroll
    for (int i = 0; i < EPL; ++i)
        if (lane * EPL + i == e) mine = s[i];
    return __shfl(mine, e / EPL);
}

// Phase A for token t: writes K_t (rank order), G(t) and the token's top expert.
template <int EPL>
__device__ void route_token(const RouteParams& p, int t, int lane, int* ids, double* gout,
                            int* top1, double* sbuf) {
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
    for (int off = 1; off < p.lpg; off <<= 1) {
        const double o1 = __shfl_xor(t1, off);
        const double o2 = __shfl_xor(t2, off);
        const double n1 = fmax(t1, o1);
        const double n2 = fmax(fmin(t1, o1), fmax(t2, o2));
        t1 = n1;
        t2 = n2;
    }
    const double gscore = p.gsize >= 2 ? t1 + t2 : t1;
    const int my_group = lane_valid ? (lane * EPL) / p.gsize : kNoIdx;

    bool gsel = false;
    for (int r = 0; r < p.topk_group; ++r) {
        double v = (lane_valid && !gsel) ? gscore : -INFINITY;
        int gi = (lane_valid && !gsel) ? my_group : kNoIdx;
        wave_argmax(v, gi);
        if (my_group == gi) gsel = true;
    }

    bool chosen[EPL];
#pragma unroll
    for (int i = 0; i < EPL; ++i) chosen[i] = false;
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
        const double sv = score_of<EPL>(s, lane, ei);
        if (lane == 0) {
            ids[r] = ei;
            sbuf[r] = sv;
        }
    }
    if (lane == 0) {
        double total = 0.0;
        for (int r = 0; r < p.k; ++r) total += sbuf[r];
        int best = kNoIdx;
        double bg = -1.0;
        for (int r = 0; r < p.k; ++r) {
            const double g = sbuf[r] / total;
            gout[r] = g;
            if (g > bg || (g == bg && ids[r] < best)) {
                bg = g;
                best = ids[r];
            }
        }
        *top1 = best;
    }
}

// Phase C for token t: K_final = (K_t ∩ A_trans) refilled from A_trans \ K_t.
template <int EPL>
__device__ void compensate_token(const RouteParams& p, int t, int lane, const int* orig,
                                 const uint8_t* trans, int* fin, double* sbuf, int* n_refill,
                                 int* n_pad) {
    double s[EPL], key[EPL];
    load_scores<EPL>(p, t, lane, s, key);
    bool in_k[EPL], tr[EPL], take[EPL], fin_f[EPL], out_f[EPL];
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
        const int e = lane * EPL + i;
        in_k[i] = false;
        for (int r = 0; r < p.k; ++r) in_k[i] |= (orig[r] == e);
        tr[i] = e < p.E && trans[e];
        take[i] = false;
        out_f[i] = false;
    }
    int n_keep = 0;
    for (int r = 0; r < p.k; ++r) n_keep += trans[orig[r]] ? 1 : 0;

    int got = 0;
    for (int r = 0; r < p.k - n_keep; ++r) {
        double v = -INFINITY;
        int ei = kNoIdx;
#pragma unroll
        for (int i = 0; i < EPL; ++i) {
            if (tr[i] && !in_k[i] && !take[i] && key[i] > v) {
                v = key[i];
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
    for (int i = 0; i < EPL; ++i) fin_f[i] = (in_k[i] && tr[i]) || take[i];

    const int m = n_keep + got;
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
        const double sv = score_of<EPL>(s, lane, ei);
        if (lane == 0) {
            fin[r] = ei;
            sbuf[r] = sv;
        }
    }
    if (lane == 0) {
        double total = 0.0;
        for (int r = 0; r < m; ++r) total += sbuf[r];
        for (int r = 0; r < p.k; ++r) {
            const size_t o = (size_t)t * p.k + r;
            if (r < m) {
                p.topk_ids[o] = fin[r];
                p.topk_w[o] = (float)(p.rs * (sbuf[r] / total));
            } else {
                fin[r] = -1;
                p.topk_ids[o] = -1;
                p.topk_w[o] = 0.0f;
            }
        }
        atomicAdd(n_refill, got);
        atomicAdd(n_pad, p.k - m);
    }
}

template <int EPL>
__global__ __launch_bounds__(kRouteThreads) void k_route_fused(RouteParams p) {
    __shared__ int s_orig[kFusedMaxT * kMaxK];
    __shared__ double s_g[kFusedMaxT * kMaxK];
    __shared__ int s_fin[kFusedMaxT * kMaxK];
    __shared__ int s_top1[kFusedMaxT];
    __shared__ double s_sbuf[kRouteWaves][kMaxK];
    __shared__ unsigned long long s_imp[kMaxE];
    __shared__ uint8_t s_act[kMaxE], s_must[kMaxE], s_prom[kMaxE], s_trans[kMaxE];
    __shared__ float s_cost[kMaxE];
    __shared__ int s_bin[kMaxE];
    __shared__ int s_sorted[kMaxE];
    __shared__ double s_mload[kMaxBins];
    __shared__ double s_fbase;
    __shared__ int s_counts[4];   // candidates, refilled slots, empty slots
    __shared__ int s_cnt[kMaxE + kMaxShared];
    __shared__ int s_off[kMaxE + kMaxShared + 1];

    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wave = tid / kWave;
    const int T = p.T, E = p.E, k = p.k;

    if (p.do_route) {
        for (int t = wave; t < T; t += kRouteWaves)
            route_token<EPL>(p, t, lane, &s_orig[t * k], &s_g[t * k], &s_top1[t], s_sbuf[wave]);
        for (int e = tid; e < E; e += kRouteThreads) {
            s_imp[e] = 0ull;
            s_act[e] = s_must[e] = s_prom[e] = 0;
            s_cost[e] = p.cost[e];
            s_bin[e] = p.bin ? p.bin[e] : 0;
        }
        if (tid < 4) s_counts[tid] = 0;
        __syncthreads();

        // Step 1: A_act, I(e) = max gate weight, A_must (threshold + each token's top expert).
        for (int i = tid; i < T * k; i += kRouteThreads) {
            const int e = s_orig[i];
            const double g = s_g[i];
            atomicMax(&s_imp[e], (unsigned long long)__double_as_longlong(g));
            s_act[e] = 1;
            if (g >= p.tau) s_must[e] = 1;
            if (p.orig_ids) p.orig_ids[i] = e;
        }
        for (int t = tid; t < T; t += kRouteThreads) s_must[s_top1[t]] = 1;
        __syncthreads();

        // Step 2: per-bin loads of A_act and A_must (ascending expert order).
        for (int b = tid; b < p.n_bins; b += kRouteThreads) {
            double la = 0.0, lm = 0.0;
            for (int e = 0; e < E; ++e) {
                if (s_bin[e] != b) continue;
                if (s_act[e]) la += (double)s_cost[e];
                if (s_must[e]) lm += (double)s_cost[e];
            }
            s_mload[b] = lm;
            if (p.bin_loads) {
                p.bin_loads[b] = la;
                p.bin_loads[p.n_bins + b] = lm;
            }
        }
        // Candidate visiting order: importance descending, index ascending.
        for (int e = tid; e < E; e += kRouteThreads) {
            if (s_act[e] && !s_must[e]) {
                const unsigned long long ie = s_imp[e];
                int rank = 0;
                for (int o = 0; o < E; ++o) {
                    if (s_act[o] && !s_must[o]) {
                        const unsigned long long io = s_imp[o];
                        rank += (io > ie || (io == ie && o < e)) ? 1 : 0;
                    }
                }
                s_sorted[rank] = e;
                atomicAdd(&s_counts[0], 1);
            }
        }
        __syncthreads();
        if (tid == 0) {
            double fb = 0.0;
            for (int b = 0; b < p.n_bins; ++b) fb = fmax(fb, s_mload[b]);
            s_fbase = fb;
        }
        __syncthreads();

        // Step 3: cost-invariant expansion, one bin per thread (bins are independent).
        const int n_cand = s_counts[0];
        for (int b = tid; b < p.n_bins; b += kRouteThreads) {
            double load = s_mload[b];
            for (int r = 0; r < n_cand; ++r) {
                const int e = s_sorted[r];
                if (s_bin[e] != b) continue;
                const double c = (double)s_cost[e];
                if (load + c <= s_fbase) {
                    s_prom[e] = 1;
                    load += c;
                }
            }
            if (p.bin_loads) p.bin_loads[2 * p.n_bins + b] = load;
        }
        __syncthreads();
        // Step 4: A_trans = A_must + promoted.
        for (int e = tid; e < E; e += kRouteThreads) s_trans[e] = s_must[e] | s_prom[e];
        __syncthreads();

        if (p.masks) {
            const int words = (E + 31) / 32;
            for (int w = tid; w < words; w += kRouteThreads) {
                uint32_t act = 0, must = 0, trans = 0, pruned = 0;
                for (int j = 0; j < 32 && w * 32 + j < E; ++j) {
                    const int e = w * 32 + j;
                    act |= (uint32_t)s_act[e] << j;
                    must |= (uint32_t)s_must[e] << j;
                    trans |= (uint32_t)s_trans[e] << j;
                    pruned |= (uint32_t)(s_act[e] && !s_trans[e]) << j;
                }
                p.masks[w] = act;
                p.masks[words + w] = must;
                p.masks[2 * words + w] = trans;
                p.masks[3 * words + w] = pruned;
            }
        }

        // Phase C: compensation.
        for (int t = wave; t < T; t += kRouteWaves)
            compensate_token<EPL>(p, t, lane, &s_orig[t * k], s_trans, &s_fin[t * k], s_sbuf[wave],
                                  &s_counts[1], &s_counts[2]);
        __syncthreads();

        if (p.stats && wave == 0) {
            int n_act = 0, n_must = 0, n_prom = 0, n_pruned = 0, n_trans = 0;
            for (int base = 0; base < E; base += kWave) {
                const int e = base + lane;
                const bool v = e < E;
                n_act += __popcll(__ballot(v && s_act[e]));
                n_must += __popcll(__ballot(v && s_must[e]));
                n_prom += __popcll(__ballot(v && s_prom[e]));
                n_pruned += __popcll(__ballot(v && s_act[e] && !s_trans[e]));
                n_trans += __popcll(__ballot(v && s_trans[e]));
            }
            if (lane == 0) {
                p.stats[0] = n_act;
                p.stats[1] = n_must;
                p.stats[2] = s_counts[0];
                p.stats[3] = n_prom;
                p.stats[4] = n_pruned;
                p.stats[5] = n_trans;
                p.stats[6] = s_counts[1];
                p.stats[7] = s_counts[2];
            }
        }
    } else {
        // Caller-supplied ids: anything outside [0, E) is an empty slot.
        for (int i = tid; i < T * k; i += kRouteThreads) {
            const int e = p.topk_ids[i];
            s_fin[i] = (e >= 0 && e < E) ? e : -1;
        }
        __syncthreads();
    }

    if (!p.do_permute) return;

    // Permutation: rows of expert slot x (x < E routed, E+s shared) are
    // [off[x], off[x+1]), tokens ascending within a slot.
    const int nx = E + p.n_shared;
    const int slots = k + p.n_shared;
    for (int x = tid; x < nx; x += kRouteThreads) s_cnt[x] = x < E ? 0 : T;
    __syncthreads();
    for (int i = tid; i < T * k; i += kRouteThreads) {
        const int e = s_fin[i];
        if (e >= 0) atomicAdd(&s_cnt[e], 1);
    }
    __syncthreads();
    if (wave == 0) {
        const int per = (nx + kWave - 1) / kWave;
        const int lo = lane * per;
        const int hi = min(lo + per, nx);
        int sum = 0, csum = 0;
        for (int x = lo; x < hi; ++x) {
            sum += s_cnt[x];
            csum += (s_cnt[x] + kChunkTokens - 1) / kChunkTokens;
        }
        int inc = sum, cinc = csum;
        for (int off = 1; off < kWave; off <<= 1) {
            const int o = __shfl_up(inc, off);
            const int co = __shfl_up(cinc, off);
            if (lane >= off) {
                inc += o;
                cinc += co;
            }
        }
        int run = inc - sum, crun = cinc - csum;
        for (int x = lo; x < hi; ++x) {
            const int cnt = s_cnt[x];
            s_off[x] = run;
            p.perm_off[x] = run;
            for (int c = 0; c * kChunkTokens < cnt; ++c) {
                int* ch = p.chunks + 4 * (crun + c);
                ch[0] = x;
                ch[1] = run + c * kChunkTokens;
                ch[2] = min(kChunkTokens, cnt - c * kChunkTokens);
                ch[3] = 0;
            }
            run += cnt;
            crun += (cnt + kChunkTokens - 1) / kChunkTokens;
        }
        const int total = __shfl(inc, kWave - 1);
        const int ctotal = __shfl(cinc, kWave - 1);
        if (lane == 0) {
            s_off[nx] = total;
            p.perm_off[nx] = total;
            *p.n_chunks = ctotal;
        }
    }
    __syncthreads();
    for (int x = tid; x < nx; x += kRouteThreads) {
        int pos = s_off[x];
        if (x < E) {
            if (s_cnt[x] == 0) continue;
            for (int t = 0; t < T; ++t) {
                for (int j = 0; j < k; ++j) {
                    if (s_fin[t * k + j] == x) {
                        p.perm_tok[pos] = t;
                        p.perm_pos[t * slots + j] = pos;
                        ++pos;
                    }
                }
            }
        } else {
            for (int t = 0; t < T; ++t) {
                p.perm_tok[pos + t] = t;
                p.perm_pos[t * slots + k + (x - E)] = pos + t;
            }
        }
    }
    for (int i = tid; i < T * k; i += kRouteThreads)
        if (s_fin[i] < 0) p.perm_pos[(i / k) * slots + (i % k)] = -1;
}

}  // namespace

hipError_t launch_route(const RouteParams& p, hipStream_t s) {
    switch (p.epl) {
        case 1: hipLaunchKernelGGL(k_route_fused<1>, dim3(1), dim3(kRouteThreads), 0, s, p); break;
        case 2: hipLaunchKernelGGL(k_route_fused<2>, dim3(1), dim3(kRouteThreads), 0, s, p); break;
        case 4: hipLaunchKernelGGL(k_route_fused<4>, dim3(1), dim3(kRouteThreads), 0, s, p); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace caee
