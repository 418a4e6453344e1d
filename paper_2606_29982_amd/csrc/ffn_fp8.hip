// 8-bit expert FFN for gfx950: OCP E4M3 weights with fp32 128x128 block
// scales, activations quantised per token per 128 channels (x before the
// gate/up products, the SwiGLU rows before the down product).
//
// One 16x16x128 MFMA consumes exactly one 128-wide scale block of the
// contraction, so each block's fp32 partial is multiplied by
// (weight-block scale) x (token-block scale) and added to the accumulator.
// Work decomposition, tiled weight layout and the deterministic split-K
// reduction are those of the 16-bit kernels.
#include <math.h>

#include "caee_internal.h"
#include "ffn_stage.h"
#include "fp8_codec.h"

namespace caee {
namespace {

typedef int i32x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kScaleOne = 127;   // E8M0 exponent of 1.0 for the MFMA's own block scales

// Per-row, per-128-column quantisation of one block of 128 values by one
// wavefront (two per lane): scale = amax / 448 (1 for an all-zero block),
// code = e4m3(value / scale), all in fp32.
__device__ inline void quant_block(const void* src, int src_bf16, long long row, int blk, int cols, uint8_t* q,
                                   float* scale, long long srow, long long sblk, int lane) {
    const long long base = row * cols + blk * 128 + 2 * lane;
    float v0, v1;
    if (src_bf16) {
        const uint32_t u = *(const uint32_t*)((const uint16_t*)src + base);
        v0 = __uint_as_float(u << 16);
        v1 = __uint_as_float(u & 0xFFFF0000u);
    } else {
        const float2 f = *(const float2*)((const float*)src + base);
        v0 = f.x;
        v1 = f.y;
    }
    float amax = fmaxf(fabsf(v0), fabsf(v1));
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) amax = fmaxf(amax, __shfl_xor(amax, off));
    const float sc = amax > 0.0f ? amax / kE4M3Max : 1.0f;
    *(uint16_t*)(q + base) = (uint16_t)e4m3_code2(v0 / sc, v1 / sc);
    if (lane == 0) scale[row * srow + blk * sblk] = sc;
}

// All blocks of `rows` consecutive rows, one wavefront per block.
__global__ __launch_bounds__(256) void k_quant_rows(const void* src, int src_bf16, long long rows, int cols,
                                                    uint8_t* q, float* scale) {
    const int lane = threadIdx.x & (kWave - 1);
    const long long w = (long long)blockIdx.x * 4 + threadIdx.x / kWave;
    const int nblk = cols / 128;
    if (w >= rows * nblk) return;
    const long long row = w / nblk;
    quant_block(src, src_bf16, row, (int)(w - row * nblk), cols, q, scale, nblk, 1, lane);
}

// The fp32 SwiGLU rows of the chunks of one work list (at most rows_max
// rows per chunk), so that each list's chain can run on its own stream.
// Scales go to hs ([row][block]), or transposed to hst ([block][row]) for
// the 8-bit GEMM.
__global__ __launch_bounds__(256) void k_quant_list(FfnParams p, int rows_max, int transposed) {
    const int lane = threadIdx.x & (kWave - 1);
    const int nblk = p.f / 128;
    const long long per_chunk = (long long)rows_max * nblk;
    const long long total = ffn_list_size(p) * per_chunk;
    for (long long w = (long long)blockIdx.x * 4 + threadIdx.x / kWave; w < total; w += (long long)gridDim.x * 4) {
        const int c = (int)(w / per_chunk);
        const int rem = (int)(w - c * per_chunk);
        const int r = rem / nblk;
        const ChunkRef ck = ffn_chunk(p, c);
        if (r >= ck.ntok) continue;
        if (transposed) quant_block(p.h, 0, ck.row0 + r, rem - r * nblk, p.f, p.hq, p.hst, 1, p.P, lane);
        else quant_block(p.h, 0, ck.row0 + r, rem - r * nblk, p.f, p.hq, p.hs, nblk, 1, lane);
    }
}

__device__ inline i32x8_t join(const u32x4_t& lo, const u32x4_t& hi) {
    return i32x8_t{(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3], (int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
}

// Contraction of one 16-row tile against up to NB 16-token blocks over
// `nblocks` 128-wide blocks.  a[m]: this lane's first weight piece (the two
// pieces of a block are `astep` apart, blocks 2*astep apart); b[tb]: the
// token row's first piece (4 pieces = 64 bytes per step); wsc[m][kb] and
// xsc[tb][kb]: block scales.  Weights are loaded U blocks ahead.
template <int U, int NA, int NB>
__device__ inline void contract_fp8(const u32x4_t* const (&a)[NA], int astep, const u32x4_t* const (&b)[NB],
                                    const float* const (&wsc)[NA], const float* const (&xsc)[NB], int nb,
                                    int nblocks, f32x4_t (&acc)[NA][NB]) {
    // Blocks past the end of the row (when nblocks is not a multiple of U)
    // are neither loaded nor multiplied.
    u32x4_t cur[NA][U][2], nxt[NA][U][2];
#pragma unroll
    for (int m = 0; m < NA; ++m)
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int h = 0; h < 2; ++h)
                cur[m][u][h] = u < nblocks ? __builtin_nontemporal_load(a[m] + (size_t)astep * (2 * u + h))
                                           : u32x4_t{0u, 0u, 0u, 0u};
    const f32x4_t zero = {0.f, 0.f, 0.f, 0.f};
    for (int kb = 0; kb < nblocks; kb += U) {
        const bool more = kb + U < nblocks;
        if (more) {
#pragma unroll
            for (int m = 0; m < NA; ++m)
#pragma unroll
                for (int u = 0; u < U; ++u)
#pragma unroll
                    for (int h = 0; h < 2; ++h)
                        nxt[m][u][h] = kb + U + u < nblocks
                                           ? __builtin_nontemporal_load(a[m] + (size_t)astep * (2 * (kb + U + u) + h))
                                           : u32x4_t{0u, 0u, 0u, 0u};
        }
        float ws[NA][U];
#pragma unroll
        for (int m = 0; m < NA; ++m)
#pragma unroll
            for (int u = 0; u < U; ++u) ws[m][u] = kb + u < nblocks ? wsc[m][kb + u] : 0.0f;
#pragma unroll
        for (int tb = 0; tb < NB; ++tb) {
            if (tb < nb) {
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    if (kb + u >= nblocks) break;
                    const int st = 2 * (kb + u);
                    const i32x8_t bv = join(b[tb][4 * st], b[tb][4 * (st + 1)]);
                    const float xs = xsc[tb][kb + u];
#pragma unroll
                    for (int m = 0; m < NA; ++m) {
                        const f32x4_t part = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(
                            join(cur[m][u][0], cur[m][u][1]), bv, zero, 0, 0, 0, kScaleOne, 0, kScaleOne);
                        acc[m][tb] += part * (ws[m][u] * xs);
                    }
                }
            }
        }
        if (more) {
#pragma unroll
            for (int m = 0; m < NA; ++m)
#pragma unroll
                for (int u = 0; u < U; ++u)
#pragma unroll
                    for (int h = 0; h < 2; ++h) cur[m][u][h] = nxt[m][u][h];
        }
    }
}

__device__ inline float silu_mul(float g, float u) { return g / (1.0f + __expf(-g)) * u; }

// Gate/up + SwiGLU, fp32 output rows (quantised afterwards).
template <int NB>
__global__ __launch_bounds__(kFfnThreads) void k_gate_up_fp8(FfnParams p) {
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
    const size_t row_units = (size_t)p.d / 16;     // 16-byte pieces per weight / x row
    const size_t ksteps = row_units / 4;            // 64-byte steps per row
    const int kblocks = p.d / 128;
    const int kper = kblocks / S;
    const size_t expert_bytes = (size_t)2 * p.f * p.d;
    const int sblk = p.d / 128;                     // scale blocks per row
    const int sp = wave % S;

    for (int item = blockIdx.x; item < total; item += gridDim.x) {
        const int c = item / items_per_chunk;
        const int jt = (item - c * items_per_chunk) * tiles_per_item + wave / S;
        const ChunkRef ck = ffn_chunk(p, c);
        const int xs_ = ck.xs, row0 = ck.row0, ntok = ck.ntok;
        const int nb = (ntok + 15) >> 4;
        const int kb0 = sp * kper;
        const u32x4_t* wb = (const u32x4_t*)ffn_weights(p, xs_, false, expert_bytes);
        const u32x4_t* const a[2] = {
            p.tiled ? wb + ((size_t)jt * ksteps + 2 * (size_t)kb0) * 64 + lane
                    : wb + (size_t)(jt * 16 + r) * row_units + g + 8 * (size_t)kb0,
            p.tiled ? wb + ((size_t)(tiles + jt) * ksteps + 2 * (size_t)kb0) * 64 + lane
                    : wb + (size_t)(p.f + jt * 16 + r) * row_units + g + 8 * (size_t)kb0};
        const int astep = p.tiled ? 64 : 4;
        const float* sbase = ffn_scales(p, xs_, false, (size_t)(2 * p.f / 128) * sblk);
        const float* const wsc[2] = {sbase + (size_t)((jt * 16) / 128) * sblk + kb0,
                                     sbase + (size_t)((p.f + jt * 16) / 128) * sblk + kb0};
        const u32x4_t* xb[NB];
        const float* xsc[NB];
#pragma unroll
        for (int tb = 0; tb < NB; ++tb) {
            int n = tb * 16 + r;
            n = (tb < nb && n < ntok) ? n : 0;   // padded token columns read a valid row; results dropped
            const int tok = ffn_token(p, xs_, row0 + n);
            xb[tb] = (const u32x4_t*)p.xq + (size_t)tok * row_units + g + 8 * (size_t)kb0;
            xsc[tb] = p.xs + (size_t)tok * sblk + kb0;
        }
        f32x4_t acc[2][NB];
#pragma unroll
        for (int m = 0; m < 2; ++m)
#pragma unroll
            for (int tb = 0; tb < NB; ++tb) acc[m][tb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        contract_fp8<kFp8U, 2, NB>(a, astep, xb, wsc, xsc, nb, kper, acc);

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
        if (sp == 0) {
            const int col = jt * 16 + 4 * g;
#pragma unroll
            for (int tb = 0; tb < NB; ++tb) {
                const int n = tb * 16 + r;
                if (tb < nb && n < ntok) {
                    float h[4];
#pragma unroll
                    for (int v = 0; v < 4; ++v) h[v] = silu_mul(acc[0][tb][v], acc[1][tb][v]);
                    *(float4*)((float*)p.h + (size_t)(row0 + n) * p.f + col) = make_float4(h[0], h[1], h[2], h[3]);
                }
            }
        }
    }
}

// Down products from the quantised SwiGLU rows.
template <int NB>
__global__ __launch_bounds__(kFfnThreads) void k_down_fp8(FfnParams p) {
    const int lane = threadIdx.x & (kWave - 1);
    const int r = lane & 15, g = lane >> 4;
    const int gw = blockIdx.x * (kFfnThreads / kWave) + (threadIdx.x / kWave);
    const int nw = gridDim.x * (kFfnThreads / kWave);
    const int tiles = p.d / 16;
    const int n_chunks = ffn_list_size(p);
    const int total = n_chunks * tiles;
    const size_t row_units = (size_t)p.f / 16;
    const size_t ksteps = row_units / 4;
    const int kblocks = p.f / 128;
    const size_t expert_bytes = (size_t)p.d * p.f;
    const int sblk = p.f / 128;

    for (int item = gw; item < total; item += nw) {
        const int c = item / tiles, it = item - c * tiles;
        const ChunkRef ck = ffn_chunk(p, c);
        const int xs_ = ck.xs, row0 = ck.row0, ntok = ck.ntok;
        const int nb = (ntok + 15) >> 4;
        const u32x4_t* wb = (const u32x4_t*)ffn_weights(p, xs_, true, expert_bytes);
        const u32x4_t* const a[1] = {p.tiled ? wb + (size_t)it * ksteps * 64 + lane
                                             : wb + (size_t)(it * 16 + r) * row_units + g};
        const int astep = p.tiled ? 64 : 4;
        const float* sbase = ffn_scales(p, xs_, true, (size_t)(p.d / 128) * sblk);
        const float* const wsc[1] = {sbase + (size_t)((it * 16) / 128) * sblk};
        const u32x4_t* hb[NB];
        const float* hsc[NB];
#pragma unroll
        for (int tb = 0; tb < NB; ++tb) {
            int n = tb * 16 + r;
            n = (tb < nb && n < ntok) ? n : 0;
            hb[tb] = (const u32x4_t*)p.hq + (size_t)(row0 + n) * row_units + g;
            hsc[tb] = p.hs + (size_t)(row0 + n) * sblk;
        }
        f32x4_t acc[1][NB];
#pragma unroll
        for (int tb = 0; tb < NB; ++tb) acc[0][tb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        contract_fp8<kFp8U, 1, NB>(a, astep, hb, wsc, hsc, nb, kblocks, acc);
#pragma unroll
        for (int tb = 0; tb < NB; ++tb) {
            const int n = tb * 16 + r;
            if (tb < nb && n < ntok) {
                store_y4(p, (size_t)(row0 + n), it * 16 + 4 * g, acc[0][tb][0], acc[0][tb][1], acc[0][tb][2],
                         acc[0][tb][3]);
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Big chunks: a stage is two 128-wide blocks of each token row, staged in
// LDS once per workgroup (the layout of ffn_stage.h: block u of the stage is
// steps 2u and 2u+1, lane l's fragment is its piece of both), together with
// the rows' two block scales.  Blocks past the end of a row (an odd number of
// blocks) are neither loaded nor multiplied.
template <int NA, int NB>
__device__ inline void big_contract_fp8(u32x4_t (*sb)[NB][kStageSteps][kWave], float (*sx)[16 * NB][2],
                                        const u32x4_t* const (&a)[NA], int astep, const float* const (&wsc)[NA],
                                        const u32x4_t* const (&rows)[NB], const float* const (&rsc)[NB], int nb,
                                        int nblocks, f32x4_t (&acc)[NA][NB]) {
    const int tid = threadIdx.x, lane = tid & (kWave - 1), r = lane & 15;
    const int nkb = (nblocks + 1) / 2;
    const int row_pieces = nblocks * 8;
    const int q = tid & (kStagePieces - 1), tl = tid >> 4;
    RowStage<NB> st;
    st.init(rows, tid);
    u32x4_t bv[NB];
    float sv[NB][2];
    u32x4_t cur[NA][2][2], nxt[NA][2][2];
    const f32x4_t zero = {0.f, 0.f, 0.f, 0.f};
    auto load_scales = [&](int kb) {
#pragma unroll
        for (int j = 0; j < NB; ++j)
            if (j < nb && q == 0) {
                sv[j][0] = rsc[j][2 * kb];
                sv[j][1] = 2 * kb + 1 < nblocks ? rsc[j][2 * kb + 1] : 0.0f;
            }
    };
    auto store_scales = [&](float (*dst)[2]) {
#pragma unroll
        for (int j = 0; j < NB; ++j)
            if (j < nb && q == 0) {
                dst[tl + 16 * j][0] = sv[j][0];
                dst[tl + 16 * j][1] = sv[j][1];
            }
    };
    auto load_a = [&](u32x4_t (&dst)[NA][2][2], int kb) {
#pragma unroll
        for (int m = 0; m < NA; ++m)
#pragma unroll
            for (int u = 0; u < 2; ++u)
#pragma unroll
                for (int h = 0; h < 2; ++h)
                    dst[m][u][h] = 2 * kb + u < nblocks
                                       ? __builtin_nontemporal_load(a[m] + (size_t)astep * (2 * (2 * kb + u) + h))
                                       : u32x4_t{0u, 0u, 0u, 0u};
    };
    st.load(bv, 0, nb, row_pieces);
    load_scales(0);
    load_a(cur, 0);
    st.store(sb[0], bv, tid, nb, 0, row_pieces);
    store_scales(sx[0]);
    __syncthreads();
    for (int kb = 0; kb < nkb; ++kb) {
        const bool more = kb + 1 < nkb;
        if (more) {
            st.load(bv, kb + 1, nb, row_pieces);
            load_scales(kb + 1);
            load_a(nxt, kb + 1);
        }
        u32x4_t (*cb)[kStageSteps][kWave] = sb[kb & 1];
        float (*cs)[2] = sx[kb & 1];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            if (2 * kb + u >= nblocks) break;
            float ws[NA];
#pragma unroll
            for (int m = 0; m < NA; ++m) ws[m] = wsc[m][2 * kb + u];
#pragma unroll
            for (int tb = 0; tb < NB; ++tb) {
                if (tb < nb) {
                    const i32x8_t b = join(cb[tb][2 * u][lane], cb[tb][2 * u + 1][lane]);
                    const float xsv = cs[16 * tb + r][u];
#pragma unroll
                    for (int m = 0; m < NA; ++m) {
                        const f32x4_t part = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(
                            join(cur[m][u][0], cur[m][u][1]), b, zero, 0, 0, 0, kScaleOne, 0, kScaleOne);
                        acc[m][tb] += part * (ws[m] * xsv);
                    }
                }
            }
        }
        if (more) {
            st.store(sb[(kb + 1) & 1], bv, tid, nb, kb + 1, row_pieces);
            store_scales(sx[(kb + 1) & 1]);
#pragma unroll
            for (int m = 0; m < NA; ++m)
#pragma unroll
                for (int u = 0; u < 2; ++u)
#pragma unroll
                    for (int h = 0; h < 2; ++h) cur[m][u][h] = nxt[m][u][h];
        }
        __syncthreads();
    }
}

#ifndef CAEE_FP8_BIG_TW_GU
#define CAEE_FP8_BIG_TW_GU 1
#endif
#ifndef CAEE_FP8_BIG_TW_DN
#define CAEE_FP8_BIG_TW_DN 2
#endif

// Gate/up of big chunks: 4 * kTW adjacent 16-feature tiles of one chunk per
// workgroup item, kTW per wave, over the whole contraction; fp32 rows out.
template <int NB>
__global__ __launch_bounds__(kFfnThreads) void k_gate_up_fp8_big(FfnParams p) {
    constexpr int kWaves = kFfnThreads / kWave;
    constexpr int kTW = CAEE_FP8_BIG_TW_GU;
    __shared__ u32x4_t s_b[2][NB][kStageSteps][kWave];
    __shared__ float s_x[2][16 * NB][2];
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    const int r = lane & 15, g = lane >> 4;
    const int tiles = p.f / 16;
    const int n_chunks = ffn_list_size(p);
    const int items_per_chunk = tiles / (kWaves * kTW);
    const int total = n_chunks * items_per_chunk;
    const size_t row_units = (size_t)p.d / 16;
    const size_t ksteps = row_units / 4;
    const int kblocks = p.d / 128;
    const size_t expert_bytes = (size_t)2 * p.f * p.d;
    const int sblk = p.d / 128;
    for (int item = blockIdx.x; item < total; item += gridDim.x) {
        const int c = item / items_per_chunk;
        const int jt0 = ((item - c * items_per_chunk) * kWaves + wave) * kTW;
        const ChunkRef ck = ffn_chunk(p, c);
        const int xs_ = ck.xs, row0 = ck.row0, ntok = ck.ntok;
        if (ffn_skip(p, xs_)) continue;   // uniform over the workgroup
        const int nb = (ntok + 15) >> 4;
        const u32x4_t* wb = (const u32x4_t*)ffn_weights(p, xs_, false, expert_bytes);
        const float* sbase = ffn_scales(p, xs_, false, (size_t)(2 * p.f / 128) * sblk);
        // Fragments 2m and 2m+1: gate and up rows of feature tile jt0 + m.
        const u32x4_t* a[2 * kTW];
        const float* wsc[2 * kTW];
#pragma unroll
        for (int m = 0; m < kTW; ++m) {
            const int jt = jt0 + m;
            a[2 * m] = p.tiled ? wb + (size_t)jt * ksteps * 64 + lane : wb + (size_t)(jt * 16 + r) * row_units + g;
            a[2 * m + 1] = p.tiled ? wb + (size_t)(tiles + jt) * ksteps * 64 + lane
                                   : wb + (size_t)(p.f + jt * 16 + r) * row_units + g;
            wsc[2 * m] = sbase + (size_t)((jt * 16) / 128) * sblk;
            wsc[2 * m + 1] = sbase + (size_t)((p.f + jt * 16) / 128) * sblk;
        }
        const u32x4_t* rows[NB];
        const float* rsc[NB];
#pragma unroll
        for (int j = 0; j < NB; ++j) {
            int n = (tid >> 4) + 16 * j;
            n = n < ntok ? n : 0;   // padded token columns read a valid row; results dropped
            const int tok = ffn_token(p, xs_, row0 + n);
            rows[j] = (const u32x4_t*)p.xq + (size_t)tok * row_units;
            rsc[j] = p.xs + (size_t)tok * sblk;
        }
        f32x4_t acc[2 * kTW][NB];
#pragma unroll
        for (int m = 0; m < 2 * kTW; ++m)
#pragma unroll
            for (int tb = 0; tb < NB; ++tb) acc[m][tb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        big_contract_fp8<2 * kTW, NB>(s_b, s_x, a, p.tiled ? 64 : 4, wsc, rows, rsc, nb, kblocks, acc);
#pragma unroll
        for (int m = 0; m < kTW; ++m) {
            const int col = (jt0 + m) * 16 + 4 * g;
#pragma unroll
            for (int tb = 0; tb < NB; ++tb) {
                const int n = tb * 16 + r;
                if (tb < nb && n < ntok) {
                    float h[4];
#pragma unroll
                    for (int v = 0; v < 4; ++v) h[v] = silu_mul(acc[2 * m][tb][v], acc[2 * m + 1][tb][v]);
                    *(float4*)((float*)p.h + (size_t)(row0 + n) * p.f + col) = make_float4(h[0], h[1], h[2], h[3]);
                }
            }
        }
    }
}

// Down products of big chunks: 8 adjacent 16-row tiles of W2 (two per wave)
// of one chunk per workgroup item.
template <int NB>
__global__ __launch_bounds__(kFfnThreads) void k_down_fp8_big(FfnParams p) {
    constexpr int kWaves = kFfnThreads / kWave;
    constexpr int kTW = CAEE_FP8_BIG_TW_DN;
    __shared__ u32x4_t s_b[2][NB][kStageSteps][kWave];
    __shared__ float s_x[2][16 * NB][2];
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    const int r = lane & 15, g = lane >> 4;
    const int tiles = p.d / 16;
    const int n_chunks = ffn_list_size(p);
    const int items_per_chunk = tiles / (kWaves * kTW);
    const int total = n_chunks * items_per_chunk;
    const size_t row_units = (size_t)p.f / 16;
    const size_t ksteps = row_units / 4;
    const int kblocks = p.f / 128;
    const size_t expert_bytes = (size_t)p.d * p.f;
    const int sblk = p.f / 128;
    for (int item = blockIdx.x; item < total; item += gridDim.x) {
        const int c = item / items_per_chunk;
        const int it0 = ((item - c * items_per_chunk) * kWaves + wave) * kTW;
        const ChunkRef ck = ffn_chunk(p, c);
        const int xs_ = ck.xs, row0 = ck.row0, ntok = ck.ntok;
        if (ffn_skip(p, xs_)) continue;
        const int nb = (ntok + 15) >> 4;
        const u32x4_t* wb = (const u32x4_t*)ffn_weights(p, xs_, true, expert_bytes);
        const float* sbase = ffn_scales(p, xs_, true, (size_t)(p.d / 128) * sblk);
        const u32x4_t* a[kTW];
        const float* wsc[kTW];
#pragma unroll
        for (int m = 0; m < kTW; ++m) {
            a[m] = p.tiled ? wb + (size_t)(it0 + m) * ksteps * 64 + lane
                           : wb + (size_t)((it0 + m) * 16 + r) * row_units + g;
            wsc[m] = sbase + (size_t)(((it0 + m) * 16) / 128) * sblk;
        }
        const u32x4_t* rows[NB];
        const float* rsc[NB];
#pragma unroll
        for (int j = 0; j < NB; ++j) {
            int n = (tid >> 4) + 16 * j;
            n = n < ntok ? n : 0;
            rows[j] = (const u32x4_t*)p.hq + (size_t)(row0 + n) * row_units;
            rsc[j] = p.hs + (size_t)(row0 + n) * sblk;
        }
        f32x4_t acc[kTW][NB];
#pragma unroll
        for (int m = 0; m < kTW; ++m)
#pragma unroll
            for (int tb = 0; tb < NB; ++tb) acc[m][tb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        big_contract_fp8<kTW, NB>(s_b, s_x, a, p.tiled ? 64 : 4, wsc, rows, rsc, nb, kblocks, acc);
#pragma unroll
        for (int m = 0; m < kTW; ++m)
#pragma unroll
            for (int tb = 0; tb < NB; ++tb) {
                const int n = tb * 16 + r;
                if (tb < nb && n < ntok) {
                    store_y4(p, (size_t)(row0 + n), (it0 + m) * 16 + 4 * g, acc[m][tb][0], acc[m][tb][1],
                             acc[m][tb][2], acc[m][tb][3]);
                }
            }
    }
}

int grid_for_waves(long long waves_needed) {
    const long long wgs = (waves_needed + 3) / 4;
    const long long cap = (long long)device_cu_count() * 8;
    return (int)(wgs < 1 ? 1 : (wgs < cap ? wgs : cap));
}

}  // namespace

hipError_t launch_quant_rows(const void* src, int src_bf16, long long rows, int cols, uint8_t* q, float* scale,
                             hipStream_t s) {
    const long long waves = rows * (cols / 128);
    if (waves == 0) return hipSuccess;
    hipLaunchKernelGGL(k_quant_rows, dim3((unsigned)((waves + 3) / 4)), dim3(256), 0, s, src, src_bf16, rows, cols,
                       q, scale);
    return hipGetLastError();
}

hipError_t launch_quant_list(const FfnParams& p, int nb, int max_chunks, bool transposed, hipStream_t s) {
    const long long waves = (long long)max_chunks * 16 * nb * (p.f / 128);
    long long blocks = (waves + 3) / 4;
    const long long cap = (long long)device_cu_count() * 16;
    if (blocks > cap) blocks = cap;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(k_quant_list, dim3((unsigned)blocks), dim3(256), 0, s, p, 16 * nb, transposed ? 1 : 0);
    return hipGetLastError();
}

hipError_t launch_gate_up_fp8(const FfnParams& p, int nb, int max_chunks, hipStream_t s) {
    if (gemm_fp8_supports(p, nb)) return launch_prefill8(p, true, max_chunks, s);
    if (nb >= 4 && kBigStaged) {
        const dim3 grid(grid_for_waves((long long)max_chunks * (p.f / 16) / CAEE_FP8_BIG_TW_GU));
        if (nb == 4) hipLaunchKernelGGL(k_gate_up_fp8_big<4>, grid, dim3(kFfnThreads), 0, s, p);
        else if (nb == 8) hipLaunchKernelGGL(k_gate_up_fp8_big<8>, grid, dim3(kFfnThreads), 0, s, p);
        else return hipErrorInvalidValue;
        return hipGetLastError();
    }
    const dim3 grid(grid_for_waves((long long)max_chunks * (p.f / 16) * p.ksplit));
    switch (nb) {
        case 1: ffn_launch(k_gate_up_fp8<1>, grid, dim3(kFfnThreads), s, p); break;
        case 2: ffn_launch(k_gate_up_fp8<2>, grid, dim3(kFfnThreads), s, p); break;
        case 4: hipLaunchKernelGGL(k_gate_up_fp8<4>, grid, dim3(kFfnThreads), 0, s, p); break;
        case 8: hipLaunchKernelGGL(k_gate_up_fp8<8>, grid, dim3(kFfnThreads), 0, s, p); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_down_fp8(const FfnParams& p, int nb, int max_chunks, hipStream_t s) {
    if (gemm_fp8_supports(p, nb)) return launch_prefill8(p, false, max_chunks, s);
    if (nb >= 4 && kBigStaged) {
        const dim3 grid(grid_for_waves((long long)max_chunks * (p.d / 16) / CAEE_FP8_BIG_TW_DN));
        if (nb == 4) hipLaunchKernelGGL(k_down_fp8_big<4>, grid, dim3(kFfnThreads), 0, s, p);
        else if (nb == 8) hipLaunchKernelGGL(k_down_fp8_big<8>, grid, dim3(kFfnThreads), 0, s, p);
        else return hipErrorInvalidValue;
        return hipGetLastError();
    }
    const dim3 grid(grid_for_waves((long long)max_chunks * (p.d / 16)));
    switch (nb) {
        case 1: hipLaunchKernelGGL(k_down_fp8<1>, grid, dim3(kFfnThreads), 0, s, p); break;
        case 2: hipLaunchKernelGGL(k_down_fp8<2>, grid, dim3(kFfnThreads), 0, s, p); break;
        case 4: hipLaunchKernelGGL(k_down_fp8<4>, grid, dim3(kFfnThreads), 0, s, p); break;
        case 8: hipLaunchKernelGGL(k_down_fp8<8>, grid, dim3(kFfnThreads), 0, s, p); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace caee
