// Grouped SwiGLU expert FFN and weighted combine (the MoE output equation
// of Sec. II-A) for gfx950.
//
// Work is a device-built list of (expert slot, first permuted row, rows)
// chunks.  Each wavefront owns one 16-row weight tile of one chunk and walks
// the whole contraction dimension, so every weight byte of every selected
// expert is read from HBM exactly once per call.  Weights stream straight
// from HBM into registers with 16-byte loads; the 16x16 MFMA takes the 16
// weight rows as its M side and up to 16 tokens as its N side.  Inside one
// 16-byte load the contraction index is permuted identically for weights and
// activations (lane group g of a k-step holds elements 8g..8g+7 for bf16),
// which leaves the dot products unchanged and keeps each row's 64 bytes per
// step contiguous.
//
//   gate/up: H[row][j] = silu(W1[j] . x) * (W3[j] . x)   (rows = tokens of the chunk)
//   down:    Y[row][i] = W2[i] . H[row]                   (fp32)
//   combine: y[t] = sum_j w[t][j] Y[pos(t,j)] + sum_s Y[pos(t,k+s)]
#include "caee_internal.h"
#include "ffn_stage.h"

namespace caee {
namespace {

#include "ffn_tile.h"

#if CAEE_FFN_WAVES_PER_EU > 0
#define CAEE_FFN_BOUNDS __launch_bounds__(kFfnThreads) __attribute__((amdgpu_waves_per_eu(CAEE_FFN_WAVES_PER_EU)))
#else
#define CAEE_FFN_BOUNDS __launch_bounds__(kFfnThreads)
#endif

// Gate/up products and SwiGLU.  A workgroup item covers 4/ksplit adjacent
// 16-column tiles of one chunk; wave w takes tile w/ksplit and contraction
// range w%ksplit.  Split partial sums meet in LDS and are added in split
// order, so the result does not depend on which wave finishes first.
template <class M, int U, int NB>
__global__ CAEE_FFN_BOUNDS void k_gate_up(FfnParams p) {
    constexpr int kWaves = kFfnThreads / kWave;
    __shared__ f32x4_t s_red[kWaves][2][NB][kWave];
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int r = lane & 15, g = lane >> 4;
    const int tiles = p.f / 16;
    const int n_chunks = ffn_list_size(p);
    const int S = gate_up_split_for(n_chunks, tiles, p.ksplit);
    const int tiles_per_item = kWaves / S;
    const int items_per_chunk = tiles / tiles_per_item;
    const int total = n_chunks * items_per_chunk;
    const size_t row_units = (size_t)p.d * M::kElemBytes / 16;
    const int kper = (int)(row_units / 4) / S;
    const size_t expert_bytes = (size_t)2 * p.f * p.d * M::kElemBytes;
    const int sp = wave % S;

    for (int item = blockIdx.x; item < total; item += gridDim.x) {
        const int c = item / items_per_chunk;
        const int jt = (item - c * items_per_chunk) * tiles_per_item + wave / S;
        const ChunkRef ck = ffn_chunk(p, c);
        const int xs = ck.xs, row0 = ck.row0, ntok = ck.ntok;
        if (ffn_skip(p, xs)) continue;   // uniform over the workgroup
        const int nb = (ntok + 15) >> 4;
        const size_t k0 = (size_t)4 * sp * kper;
        const u32x4_t* wb = (const u32x4_t*)ffn_weights(p, xs, false, expert_bytes);
        const size_t ksteps = row_units / 4;
        // Tiled: block (tile, step) is 64 consecutive 16-byte pieces, one per lane.
        const u32x4_t* const a[2] = {
            p.tiled ? wb + ((size_t)jt * ksteps + (size_t)sp * kper) * 64 + lane
                    : wb + (size_t)(jt * 16 + r) * row_units + g + k0,
            p.tiled ? wb + ((size_t)(tiles + jt) * ksteps + (size_t)sp * kper) * 64 + lane
                    : wb + (size_t)(p.f + jt * 16 + r) * row_units + g + k0};
        const int astep = p.tiled ? 64 : 4;
        const u32x4_t* xb[NB];
#pragma unroll
        for (int tb = 0; tb < NB; ++tb) {
            int n = tb * 16 + r;
            n = (tb < nb && n < ntok) ? n : 0;   // padded token columns read a valid row; results dropped
            xb[tb] = (const u32x4_t*)p.x + (size_t)ffn_token(p, xs, row0 + n) * row_units + g + k0;
        }
        f32x4_t acc[2][NB];
#pragma unroll
        for (int m = 0; m < 2; ++m)
#pragma unroll
            for (int tb = 0; tb < NB; ++tb) acc[m][tb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        tile_contract<M, U, 2, NB>(a, astep, xb, nb, kper, acc);

        if (S > 1) {
#pragma unroll
            for (int m = 0; m < 2; ++m)
#pragma unroll
                for (int tb = 0; tb < NB; ++tb) s_red[wave][m][tb][lane] = acc[m][tb];
            __syncthreads();
            if (sp == 0) {
#pragma unroll
                for (int m = 0; m < 2; ++m)
#pragma unroll
                    for (int tb = 0; tb < NB; ++tb) {
                        f32x4_t sum = s_red[wave][m][tb][lane];
                        for (int q = 1; q < S; ++q) sum += s_red[wave + q][m][tb][lane];
                        acc[m][tb] = sum;
                    }
            }
            __syncthreads();
        }
        // Lane holds rows 4g..4g+3 of the tile (intermediate features) for token column r.
        if (sp == 0) {
            const int col = jt * 16 + 4 * g;
#pragma unroll
            for (int tb = 0; tb < NB; ++tb) {
                const int n = tb * 16 + r;
                if (tb < nb && n < ntok) {
                    float h[4];
#pragma unroll
                    for (int v = 0; v < 4; ++v) h[v] = silu_mul(acc[0][tb][v], acc[1][tb][v]);
                    store_h<M>(p, (size_t)(row0 + n) * p.f + col, h);
                }
            }
        }
    }
}

// Down products: Y[row][i] = W2[i] . H[row], one 16-row tile per work item.
template <class M, int U, int NB>
__global__ CAEE_FFN_BOUNDS void k_down(FfnParams p) {
    const int lane = threadIdx.x & (kWave - 1);
    const int r = lane & 15, g = lane >> 4;
    const int gw = blockIdx.x * (kFfnThreads / kWave) + (threadIdx.x / kWave);
    const int nw = gridDim.x * (kFfnThreads / kWave);
    const int tiles = p.d / 16;
    const int n_chunks = ffn_list_size(p);
    const int total = n_chunks * tiles;
    const size_t row_units = (size_t)p.f * M::kElemBytes / 16;
    const int ksteps = (int)(row_units / 4);
    const size_t expert_bytes = (size_t)p.d * p.f * M::kElemBytes;

    for (int item = gw; item < total; item += nw) {
        const int c = item / tiles, it = item - c * tiles;
        const ChunkRef ck = ffn_chunk(p, c);
        const int xs = ck.xs, row0 = ck.row0, ntok = ck.ntok;
        if (ffn_skip(p, xs)) continue;
        const int nb = (ntok + 15) >> 4;
        const u32x4_t* wb = (const u32x4_t*)ffn_weights(p, xs, true, expert_bytes);
        const u32x4_t* const a[1] = {p.tiled ? wb + (size_t)it * ksteps * 64 + lane
                                             : wb + (size_t)(it * 16 + r) * row_units + g};
        const int astep = p.tiled ? 64 : 4;
        const u32x4_t* hb[NB];
#pragma unroll
        for (int tb = 0; tb < NB; ++tb) {
            int n = tb * 16 + r;
            n = (tb < nb && n < ntok) ? n : 0;
            hb[tb] = (const u32x4_t*)p.h + (size_t)(row0 + n) * row_units + g;
        }
        f32x4_t acc[1][NB];
#pragma unroll
        for (int tb = 0; tb < NB; ++tb) acc[0][tb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        tile_contract<M, U, 1, NB, (NB <= CAEE_DOWN_AHEAD_NB)>(a, astep, hb, nb, ksteps, acc);
#pragma unroll
        for (int tb = 0; tb < NB; ++tb) {
            const int n = tb * 16 + r;
            if (tb < nb && n < ntok) {
                float* o = (float*)p.yperm + (size_t)(row0 + n) * p.d + it * 16 + 4 * g;
                *(float4*)o = make_float4(acc[0][tb][0], acc[0][tb][1], acc[0][tb][2], acc[0][tb][3]);
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Big chunks (more than 32 rows of one expert).  With many token columns per
// weight tile the activation rows, not the weights, dominate the load
// traffic: read by every wave from L2 they would cost each wave NB times its
// weight bytes.  Here a workgroup stages the chunk's rows for U contraction
// steps in LDS once (double buffered, one barrier per stage) and its four
// waves, each on its own weight tiles, read their MFMA fragments from LDS.
// LDS stage layout: [token block][step][lane] 16-byte pieces, i.e. exactly
// the B fragment of lane l (token 16*tb + l%16, bytes 16*(l/16) of the step),
// so every fragment read is one conflict-free 16-byte LDS load.

// Contraction of NA weight-tile fragments per wave against a chunk's staged
// rows over `nkb` stages of U steps.  a[m]: this lane's first weight piece of
// tile m (consecutive steps `astep` pieces apart); rows[j]: token row of
// staged block j for this thread's staging slot.
template <class M, int NA, int NB>
__device__ inline void big_contract(u32x4_t (*sb)[NB][kStageSteps][kWave], const u32x4_t* const (&a)[NA],
                                    int astep, const u32x4_t* const (&rows)[NB], int nb, int nkb,
                                    f32x4_t (&acc)[NA][NB]) {
    constexpr int U = kStageSteps;
    const int tid = threadIdx.x, lane = tid & (kWave - 1);
    const int row_pieces = nkb * kStagePieces;
    RowStage<NB> st;
    st.init(rows, tid);
    u32x4_t bv[NB];
    u32x4_t cur[NA][U], nxt[NA][U];
    st.load(bv, 0, nb, row_pieces);
#pragma unroll
    for (int m = 0; m < NA; ++m)
#pragma unroll
        for (int u = 0; u < U; ++u) cur[m][u] = __builtin_nontemporal_load(a[m] + (size_t)astep * u);
    st.store(sb[0], bv, tid, nb, 0, row_pieces);
    __syncthreads();
    for (int kb = 0; kb < nkb; ++kb) {
        const bool more = kb + 1 < nkb;
        if (more) {
            st.load(bv, kb + 1, nb, row_pieces);
#pragma unroll
            for (int m = 0; m < NA; ++m)
#pragma unroll
                for (int u = 0; u < U; ++u)
                    nxt[m][u] = __builtin_nontemporal_load(a[m] + (size_t)astep * ((kb + 1) * U + u));
        }
        u32x4_t (*cb)[U][kWave] = sb[kb & 1];
#pragma unroll
        for (int tb = 0; tb < NB; ++tb) {
            if (tb < nb) {
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const u32x4_t b = cb[tb][u][lane];
#pragma unroll
                    for (int m = 0; m < NA; ++m) M::mma(acc[m][tb], cur[m][u], b);
                }
            }
        }
        if (more) {
            st.store(sb[(kb + 1) & 1], bv, tid, nb, kb + 1, row_pieces);
#pragma unroll
            for (int m = 0; m < NA; ++m)
#pragma unroll
                for (int u = 0; u < U; ++u) cur[m][u] = nxt[m][u];
        }
        __syncthreads();
    }
}

// Gate/up of big chunks: a workgroup item is 4 adjacent 16-feature tiles of
// one chunk, one per wave, over the whole contraction.
template <class M, int NB>
__global__ __launch_bounds__(kFfnThreads) void k_gate_up_big(FfnParams p) {
    constexpr int kWaves = kFfnThreads / kWave;
    __shared__ u32x4_t s_b[2][NB][kStageSteps][kWave];
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    const int r = lane & 15, g = lane >> 4;
    const int n_chunks = ffn_list_size(p);
    const int tiles = p.f / 16;
    const int items_per_chunk = tiles / kWaves;
    const int total = n_chunks * items_per_chunk;
    const size_t row_units = (size_t)p.d * M::kElemBytes / 16;
    const int ksteps = (int)(row_units / 4);
    const size_t expert_bytes = (size_t)2 * p.f * p.d * M::kElemBytes;
    for (int item = blockIdx.x; item < total; item += gridDim.x) {
        const int c = item / items_per_chunk;
        const int jt = (item - c * items_per_chunk) * kWaves + wave;
        const ChunkRef ck = ffn_chunk(p, c);
        const int xs = ck.xs, row0 = ck.row0, ntok = ck.ntok;
        if (ffn_skip(p, xs)) continue;   // uniform over the workgroup
        const int nb = (ntok + 15) >> 4;
        const u32x4_t* wb = (const u32x4_t*)ffn_weights(p, xs, false, expert_bytes);
        const u32x4_t* const a[2] = {
            p.tiled ? wb + (size_t)jt * ksteps * 64 + lane : wb + (size_t)(jt * 16 + r) * row_units + g,
            p.tiled ? wb + (size_t)(tiles + jt) * ksteps * 64 + lane
                    : wb + (size_t)(p.f + jt * 16 + r) * row_units + g};
        const u32x4_t* rows[NB];
#pragma unroll
        for (int j = 0; j < NB; ++j) {
            int n = (tid >> 4) + 16 * j;
            n = n < ntok ? n : 0;   // padded token columns read a valid row; results dropped
            rows[j] = (const u32x4_t*)p.x + (size_t)ffn_token(p, xs, row0 + n) * row_units;
        }
        f32x4_t acc[2][NB];
#pragma unroll
        for (int m = 0; m < 2; ++m)
#pragma unroll
            for (int tb = 0; tb < NB; ++tb) acc[m][tb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        big_contract<M, 2, NB>(s_b, a, p.tiled ? 64 : 4, rows, nb, ksteps / kStageSteps, acc);
        const int col = jt * 16 + 4 * g;
#pragma unroll
        for (int tb = 0; tb < NB; ++tb) {
            const int n = tb * 16 + r;
            if (tb < nb && n < ntok) {
                float h[4];
#pragma unroll
                for (int v = 0; v < 4; ++v) h[v] = silu_mul(acc[0][tb][v], acc[1][tb][v]);
                store_h<M>(p, (size_t)(row0 + n) * p.f + col, h);
            }
        }
    }
}

// Down products of big chunks: a workgroup item is 8 adjacent 16-row tiles
// of W2 (two per wave) of one chunk.
template <class M, int NB>
__global__ __launch_bounds__(kFfnThreads) void k_down_big(FfnParams p) {
    constexpr int kWaves = kFfnThreads / kWave;
    constexpr int kTW = 2;
    __shared__ u32x4_t s_b[2][NB][kStageSteps][kWave];
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    const int r = lane & 15, g = lane >> 4;
    const int n_chunks = ffn_list_size(p);
    const int tiles = p.d / 16;
    const int items_per_chunk = tiles / (kWaves * kTW);
    const int total = n_chunks * items_per_chunk;
    const size_t row_units = (size_t)p.f * M::kElemBytes / 16;
    const int ksteps = (int)(row_units / 4);
    const size_t expert_bytes = (size_t)p.d * p.f * M::kElemBytes;
    for (int item = blockIdx.x; item < total; item += gridDim.x) {
        const int c = item / items_per_chunk;
        const int it0 = ((item - c * items_per_chunk) * kWaves + wave) * kTW;
        const ChunkRef ck = ffn_chunk(p, c);
        const int xs = ck.xs, row0 = ck.row0, ntok = ck.ntok;
        if (ffn_skip(p, xs)) continue;
        const int nb = (ntok + 15) >> 4;
        const u32x4_t* wb = (const u32x4_t*)ffn_weights(p, xs, true, expert_bytes);
        const u32x4_t* a[kTW];
#pragma unroll
        for (int m = 0; m < kTW; ++m)
            a[m] = p.tiled ? wb + (size_t)(it0 + m) * ksteps * 64 + lane
                           : wb + (size_t)((it0 + m) * 16 + r) * row_units + g;
        const u32x4_t* rows[NB];
#pragma unroll
        for (int j = 0; j < NB; ++j) {
            int n = (tid >> 4) + 16 * j;
            n = n < ntok ? n : 0;
            rows[j] = (const u32x4_t*)p.h + (size_t)(row0 + n) * row_units;
        }
        f32x4_t acc[kTW][NB];
#pragma unroll
        for (int m = 0; m < kTW; ++m)
#pragma unroll
            for (int tb = 0; tb < NB; ++tb) acc[m][tb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        big_contract<M, kTW, NB>(s_b, a, p.tiled ? 64 : 4, rows, nb, ksteps / kStageSteps, acc);
#pragma unroll
        for (int m = 0; m < kTW; ++m)
#pragma unroll
            for (int tb = 0; tb < NB; ++tb) {
                const int n = tb * 16 + r;
                if (tb < nb && n < ntok) {
                    float* o = (float*)p.yperm + (size_t)(row0 + n) * p.d + (it0 + m) * 16 + 4 * g;
                    *(float4*)o = make_float4(acc[m][tb][0], acc[m][tb][1], acc[m][tb][2], acc[m][tb][3]);
                }
            }
    }
}

// Row-major -> tiled repack, one thread per 16-byte piece of the destination.
__global__ __launch_bounds__(256) void k_pack(const u32x4_t* __restrict__ src, u32x4_t* __restrict__ dst,
                                              long long rows, long long row_units, long long count) {
    const long long per_mat = rows * row_units;
    const long long total = count * per_mat;
    const long long ksteps = row_units / 4;
    for (long long i = (long long)blockIdx.x * 256 + threadIdx.x; i < total; i += (long long)gridDim.x * 256) {
        const long long m = i / per_mat;
        const long long rem = i - m * per_mat;
        const long long blk = rem >> 6;
        const int l = (int)(rem & 63);
        const long long t = blk / ksteps, st = blk - t * ksteps;
        dst[i] = src[m * per_mat + (16 * t + (l & 15)) * row_units + 4 * st + (l >> 4)];
    }
}

// One thread per W output features of one token: 4, or 8 when the expert
// output rows are bf16 (one 16-byte load per row).  Slots are added in
// order with fp32 fused multiply-adds, then the shared experts (expert
// output rows are bf16 when W = 8, fp32 when W = 4).  The slot positions and
// weights (up to KM slots) are all loaded first, then every row, so a thread
// waits for two round trips to memory, not one per slot.
template <int W, int KM>
__global__ __launch_bounds__(256) void k_combine(FfnParams p) {
    const int per_tok = (p.d / W + 255) / 256;
    const int t = blockIdx.x / per_tok;
    const int c = ((blockIdx.x - t * per_tok) * 256 + threadIdx.x) * W;
    if (c >= p.d) return;
    const int slots = p.k + p.n_shared;
    auto load = [&](int pos, float (&v)[W]) {
        if constexpr (W == 8) {
            const uint4 pk = *(const uint4*)((const uint16_t*)p.yperm + (size_t)pos * p.d + c);
            const uint32_t u[4] = {pk.x, pk.y, pk.z, pk.w};
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                v[2 * i] = __uint_as_float(u[i] << 16);
                v[2 * i + 1] = __uint_as_float(u[i] & 0xFFFF0000u);
            }
        } else {
            const float4 f = *(const float4*)((const float*)p.yperm + (size_t)pos * p.d + c);
            v[0] = f.x;
            v[1] = f.y;
            v[2] = f.z;
            v[3] = f.w;
        }
    };
    const int32_t* pp = p.perm_pos + (size_t)t * slots;
    const float* pw = p.topk_w + (size_t)t * p.k;
    int pos[KM];
    float wt[KM];
#pragma unroll
    for (int j = 0; j < KM; ++j) {
        pos[j] = j < p.k ? pp[j] : -1;
        wt[j] = j < p.k ? pw[j] : 0.f;
    }
    // Every row load is issued (an empty slot reads row 0 and is not added).
    float v[KM][W];
#pragma unroll
    for (int j = 0; j < KM; ++j) load(pos[j] >= 0 ? pos[j] : 0, v[j]);
    float acc[W];
#pragma unroll
    for (int i = 0; i < W; ++i) acc[i] = 0.f;
#pragma unroll
    for (int j = 0; j < KM; ++j) {
#pragma unroll
        for (int i = 0; i < W; ++i) acc[i] = pos[j] >= 0 ? fmaf(wt[j], v[j][i], acc[i]) : acc[i];
    }
    float vs[W];
    for (int s = 0; s < p.n_shared; ++s) {
        load(pp[p.k + s], vs);
#pragma unroll
        for (int i = 0; i < W; ++i) acc[i] += vs[i];
    }
    const size_t o = (size_t)t * p.d + c;
#pragma unroll
    for (int i = 0; i < W; i += 4) {
        if (p.y_bf16) {
            uint2 pk;
            pk.x = bf16_rne(acc[i]) | (bf16_rne(acc[i + 1]) << 16);
            pk.y = bf16_rne(acc[i + 2]) | (bf16_rne(acc[i + 3]) << 16);
            *(uint2*)((uint16_t*)p.y + o + i) = pk;
        } else {
            *(float4*)((float*)p.y + o + i) = make_float4(acc[i], acc[i + 1], acc[i + 2], acc[i + 3]);
        }
    }
}

int grid_for(long long waves_needed) {
    const long long wgs = (waves_needed + 3) / 4;
    const long long cap = (long long)device_cu_count() * 8;
    return (int)(wgs < 1 ? 1 : (wgs < cap ? wgs : cap));
}

template <class M, template <class, int, int> class K, int U1, int U>
hipError_t launch_nb(const FfnParams& p, int nb, dim3 grid, hipStream_t s) {
    switch (nb) {
        case 1: ffn_launch(K<M, U1, 1>::run, grid, dim3(kFfnThreads), s, p); break;
        case 2: ffn_launch(K<M, U, 2>::run, grid, dim3(kFfnThreads), s, p); break;
        case 4: ffn_launch(K<M, U, 4>::run, grid, dim3(kFfnThreads), s, p); break;
        case 8: ffn_launch(K<M, U, 8>::run, grid, dim3(kFfnThreads), s, p); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <class M, int U, int NB>
struct GateUpK {
    static constexpr auto run = k_gate_up<M, U, NB>;
};
template <class M, int U, int NB>
struct DownK {
    static constexpr auto run = k_down<M, U, NB>;
};

template <class M>
hipError_t launch_big(const FfnParams& p, bool gate_up, int nb, dim3 grid, hipStream_t s) {
    switch (nb) {
        case 4:
            if (gate_up) hipLaunchKernelGGL((k_gate_up_big<M, 4>), grid, dim3(kFfnThreads), 0, s, p);
            else hipLaunchKernelGGL((k_down_big<M, 4>), grid, dim3(kFfnThreads), 0, s, p);
            break;
        case 8:
            if (gate_up) hipLaunchKernelGGL((k_gate_up_big<M, 8>), grid, dim3(kFfnThreads), 0, s, p);
            else hipLaunchKernelGGL((k_down_big<M, 8>), grid, dim3(kFfnThreads), 0, s, p);
            break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gate_up(const FfnParams& p, int w_dtype, int nb, int max_chunks, hipStream_t s) {
    if (w_dtype == CAEE_BF16 && gemm_bf16_supports(p, nb)) return launch_gemm(p, true, max_chunks, s);
    if (nb >= 4 && kBigStaged) {
        const dim3 grid(grid_for((long long)max_chunks * (p.f / 16)));
        if (w_dtype == CAEE_BF16) return launch_big<Bf16Math>(p, true, nb, grid, s);
        if (w_dtype == CAEE_F32) return launch_big<F32Math>(p, true, nb, grid, s);
        return hipErrorInvalidValue;
    }
    const dim3 grid(grid_for((long long)max_chunks * (p.f / 16) * p.ksplit));   // waves wanted
    if (w_dtype == CAEE_BF16) return launch_nb<Bf16Math, GateUpK, kGateUpU1, kGateUpU>(p, nb, grid, s);
    if (w_dtype == CAEE_F32) return launch_nb<F32Math, GateUpK, kGateUpU1, kGateUpU>(p, nb, grid, s);
    return hipErrorInvalidValue;
}

hipError_t launch_down(const FfnParams& p, int w_dtype, int nb, int max_chunks, hipStream_t s) {
    if (w_dtype == CAEE_BF16 && gemm_bf16_supports(p, nb)) return launch_gemm(p, false, max_chunks, s);
    if (nb >= 4 && kBigStaged) {
        const dim3 grid(grid_for((long long)max_chunks * (p.d / 16) / 2));
        if (w_dtype == CAEE_BF16) return launch_big<Bf16Math>(p, false, nb, grid, s);
        if (w_dtype == CAEE_F32) return launch_big<F32Math>(p, false, nb, grid, s);
        return hipErrorInvalidValue;
    }
    const dim3 grid(grid_for((long long)max_chunks * (p.d / 16)));
    if (w_dtype == CAEE_BF16) return launch_nb<Bf16Math, DownK, kDownU1, kDownU>(p, nb, grid, s);
    if (w_dtype == CAEE_F32) return launch_nb<F32Math, DownK, kDownU1, kDownU>(p, nb, grid, s);
    return hipErrorInvalidValue;
}

hipError_t launch_pack(const void* src, void* dst, long long rows, long long row_units, long long count,
                       hipStream_t s) {
    const long long total = count * rows * row_units;
    long long blocks = (total + 255) / 256;
    const long long cap = (long long)device_cu_count() * 16;
    if (blocks > cap) blocks = cap;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(k_pack, dim3((unsigned)blocks), dim3(256), 0, s, (const u32x4_t*)src, (u32x4_t*)dst, rows,
                       row_units, count);
    return hipGetLastError();
}

hipError_t launch_combine(const FfnParams& p, hipStream_t s) {
    const dim3 g8(((p.d / 8 + 255) / 256) * p.T), g4(((p.d / 4 + 255) / 256) * p.T);
    if (p.k <= 8) {
        if (p.y_half) hipLaunchKernelGGL((k_combine<8, 8>), g8, dim3(256), 0, s, p);
        else hipLaunchKernelGGL((k_combine<4, 8>), g4, dim3(256), 0, s, p);
    } else {
        if (p.y_half) hipLaunchKernelGGL((k_combine<8, kMaxK>), g8, dim3(256), 0, s, p);
        else hipLaunchKernelGGL((k_combine<4, kMaxK>), g4, dim3(256), 0, s, p);
    }
    return hipGetLastError();
}

}  // namespace caee
