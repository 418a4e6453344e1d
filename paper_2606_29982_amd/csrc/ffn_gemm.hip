// LDS-pipelined expert products for big chunks: 8-bit at prefill sizes,
// bf16 for the hot experts of decode batches.
//
// A workgroup of 8 waves computes a 256-weight-row x 128-token tile (or,
// built with CAEE_GEMM_TILES=8, 128 x 256) of one chunk over the whole
// contraction, one 128-wide block (one scaled 16x16x128
// MFMA deep) per pipeline stage.  Weights (tiled order: the 2 KB of one
// 16-row tile and one block are contiguous), the chunk's token rows and the
// rows' block scales go straight from global memory to LDS with the 16-byte
// (and 4-byte) direct-to-LDS loads of gfx950, three stages in a ring, so that
// two stages of loads are in flight while one is multiplied and no register
// holds staged data.  Every wave issues the same number of loads per stage,
// so a wave waits for its oldest stage with a constant vmcnt, and one barrier
// per stage makes all waves' loads of that stage visible.
//
// The tile is as wide in tokens as a chunk can be.  Each wave owns 4 weight
// tiles x 4 token tiles (64 x 64 outputs); two waves share a SIMD, so one
// wave's fp32 block-scale arithmetic (VALU) overlaps the other's matrix
// instructions.  With R = kTiles / 4 waves across the rows, wave
// w = R * c + q takes token tiles 4c .. 4c + 3 and
//   gate/up: features 2q, 2q + 1 of the tile's kTiles / 2 (gate and up rows
//            of each) -> SwiGLU rows (8-bit: e4m3 codes + block scales;
//            bf16: bf16);
//   down:    row tiles 4q .. 4q + 3 -> Y rows (bf16 on the 8-bit path,
//            fp32 otherwise).
// The rows' block scales are read transposed ([block][permuted row]), one
// 128-byte line per wave and block.  Measured at the 4096-token prefill, the
// 256 x 128 tile is faster than 128 x 256 (which reads each weight byte once
// for experts with up to 256 rows, but issues twice the token-row loads).
//
// The 8-bit down product runs a pair of chunks of one expert (adjacent
// pieces of a slot cut into several, at most 256 rows together) in the
// 128 x 256 shape of the same stage: half the weight tiles, twice the token
// tiles, the same six loads per wave.  Each chunk of the pair keeps its
// groups' worth of items, which take the pair's first and second half of
// the weight-row groups, so the item list stays dense, and the pair's
// weights stream once instead of once per chunk.  Gate/up stays in the
// 256 x 128 shape: its epilogue quantises whole 128-feature blocks.
#include "caee_internal.h"
#include "fp8_codec.h"

namespace caee {
namespace {

typedef int i32x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void_t;
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));

constexpr int kScaleOne = 127;        // E8M0 1.0: the MFMA's own block scales are unused
// Workgroup tile: kTiles 16-row weight tiles x kNT 16-token tiles, 8 waves
// of 4 x 4 tiles each.
#ifndef CAEE_GEMM_TILES
#define CAEE_GEMM_TILES 16
#endif
constexpr int kTiles = CAEE_GEMM_TILES;
constexpr int kNT = 128 / kTiles;
constexpr int kWaveNT = 4;            // token tiles per wave
constexpr int kRowWaves = kTiles / 4; // waves across the weight rows
static_assert(kTiles == 8 || kTiles == 16, "tile shape");
// With 256-row tiles a gate/up item holds 128 features, one quantisation
// block of each of its token rows: the epilogue quantises the SwiGLU rows
// itself (e4m3 codes and transposed block scales for the down product).
constexpr bool kFuseQuant = kTiles == 16;
// Whether the items are laid out by XCD (see the kernel; measured slower at
// the 4096-token prefill, so off by default).
#ifndef CAEE_GEMM_XCD
#define CAEE_GEMM_XCD 0
#endif
constexpr int kStages = 3;
constexpr int kGemmWaves = 8;
constexpr int kGemmThreads = kGemmWaves * kWave;
// 8-bit down items of paired chunks take the other shape of the same stage.
constexpr bool kWideDown = kTiles == 16;
// Fragments of one stage: 2 halves of every weight tile, then of every token
// tile (either shape: 2 * (16 + 8) = 2 * (8 + 16)).
constexpr int kFrags = 2 * (kTiles + kNT);
constexpr int kLoads = kTiles / 4 + kNT / 4;   // fragment loads per wave and stage, either shape

// Loads per wave and stage: the weight and token-row pieces, plus (8-bit)
// one load of the rows' block scales.
template <bool kFp8>
constexpr int loads_per_stage() { return kLoads + (kFp8 ? 1 : 0); }
constexpr int kMaxKBlocks = 128;      // contraction up to 16384
constexpr int kXcds = 8;              // accelerator complex dies, each with its own L2

struct GemmStage {
    u32x4_t f[kFrags][kWave];         // [2 * tile + half] weights, then [2 * tiles + 2 * token tile + half] rows
    float x[kGemmWaves][kWave];       // row scales: token n at [n / per][n % per], per = 2 * token tiles
};

__device__ inline i32x8_t join(const u32x4_t& lo, const u32x4_t& hi) {
    return i32x8_t{(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3], (int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
}

__device__ inline float silu_mul(float g, float u) { return g / (1.0f + __expf(-g)) * u; }


// Waits until at most n of this wave's vector memory loads are outstanding
// (gfx9 s_waitcnt: vmcnt in bits 3:0 and 15:14, expcnt and lgkmcnt not waited).
template <int N>
__device__ inline void wait_vm() {
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | (((N >> 4) & 3) << 14));
}

// Workgroup barrier without the memory fence of __syncthreads (which would
// wait for every load in flight); the empty asm keeps the compiler from
// moving memory accesses across it.
__device__ inline void stage_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// kFp8: e4m3 weights with fp32 block scales and quantised rows, one scaled
// 16x16x128 MFMA per 128-element stage; otherwise bf16 weights and rows,
// two 16x16x32 MFMAs per 64-element stage (the same 128 bytes per row).
template <bool kGateUp, bool kFp8>
__global__ __launch_bounds__(kGemmThreads) void k_gemm(FfnParams p) {
    constexpr int kLoadsPerStage = loads_per_stage<kFp8>();
    constexpr int kEb = kFp8 ? 1 : 2;                  // bytes per element
    // The ring's stages are separate LDS objects (and the code below names
    // each statically), so the compiler can tell a read of one stage from the
    // loads still filling the others and does not wait for those.
    __shared__ GemmStage st0, st1, st2;
    // Weight block scales of the item: the tile's first and second half of
    // weight rows each fall in one 128-row scale row.  Read from LDS in the
    // pipeline, as a global load there would make the wave drain its loads.
    __shared__ float wsl[2][kMaxKBlocks];
    const int tid = threadIdx.x, lane = tid & (kWave - 1);
    // Wave index as a scalar: the tile and fragment indices derived from it
    // stay in scalar registers.
    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
    const int r = lane & 15, g = lane >> 4;
    constexpr bool kWide = kWideDown && kFp8 && !kGateUp;
    const int K = kGateUp ? p.d : p.f;                 // contraction length
    const int kblocks = K * kEb / 128;                 // pipeline stages (128 bytes of each row)
    const size_t ksteps = (size_t)K * kEb / 64;        // 64-byte steps per weight row
    const size_t row_units = (size_t)K * kEb / 16;     // 16-byte pieces per token row
    const int rows_out = kGateUp ? p.f : p.d;          // features (gate/up) or output rows (down)
    const int groups = kGateUp ? rows_out / (16 * kTiles / 2) : rows_out / (16 * kTiles);
    const int n_chunks = ffn_list_size(p);
    const int total = n_chunks * groups;
    const size_t expert_bytes = (kGateUp ? (size_t)2 * p.f * p.d : (size_t)p.d * p.f) * kEb;
    const size_t scales_per_expert = (size_t)((kGateUp ? 2 * p.f : p.d) / 128) * kblocks;
    const f32x4_t zero = {0.f, 0.f, 0.f, 0.f};
    // Workgroups go to the XCDs round robin (workgroup b to XCD b % 8).  With
    // a grid that is a multiple of 8, XCD x takes the x-th eighth of the item
    // list, so the items of one chunk (same token rows, different weight
    // groups) and those of one expert's consecutive chunks (same weights) run
    // at the same time on one XCD and share its L2.
    int item = blockIdx.x, item_end = total, item_step = gridDim.x;
    if (CAEE_GEMM_XCD && gridDim.x % kXcds == 0) {
        const int x = blockIdx.x % kXcds, per = gridDim.x / kXcds;
        item = (int)((long long)x * total / kXcds) + blockIdx.x / kXcds;
        item_end = (int)((long long)(x + 1) * total / kXcds);
        item_step = per;
    }
    for (; item < item_end; item += item_step) {
        const int c = item / groups;
        const ChunkRef ck = ffn_chunk(p, c);
        const int xs = ck.xs;
        if (ffn_skip(p, xs)) continue;   // uniform over the workgroup
        int row0 = ck.row0, ntok = ck.ntok, grp = item - c * groups;
        // Paired chunk: the pair's rows, and half-group grp (first chunk of
        // the pair) or groups + grp (second).
        const bool wide = kWide && ck.pair != 0;
        if (wide) {
            const ChunkRef o = ffn_chunk(p, c + ck.pair);
            if (ck.pair < 0) {
                row0 = o.row0;
                grp += groups;
            }
            ntok += o.ntok;
        }
        // Item shape: tiles weight tiles x nts token tiles; waves rw across
        // the weight rows (4 x 4 output tiles per wave in both shapes).
        const int tiles = wide ? kTiles / 2 : kTiles, nts = wide ? 2 * kNT : kNT;
        const int rw = tiles / 4, wq = wave % rw, wc = wave / rw;   // weight rows, token columns
        const int na = tiles / 4;                          // weight fragment loads per wave (the rest: rows)
        const int bbase = 2 * tiles;                       // first token-row fragment of a stage
        const int xsh = wide ? 5 : 4;                      // log2 of the tokens per wave whose scales it loads
        const int nb = (ntok + 15) >> 4;
        const u32x4_t* wb = (const u32x4_t*)ffn_weights(p, xs, kGateUp ? false : true, expert_bytes);
        const float* wsc = kFp8 ? ffn_scales(p, xs, kGateUp ? false : true, scales_per_expert) : nullptr;
        // Expert-relative weight tile of workgroup tile slot i.
        auto tile_of = [&](int i) {
            if (kGateUp) return i < kTiles / 2 ? grp * (kTiles / 2) + i : p.f / 16 + grp * (kTiles / 2) + i - kTiles / 2;
            return grp * tiles + i;
        };
        // This wave's kLoads fragment loads per stage: (tile, half) pairs
        // j = na * w + i of the weights, then (token tile, half) pairs
        // j = (kLoads - na) * w + i of the rows; and the scales of tokens
        // per * w .. + per - 1 (the other lanes repeat them into padding).
        const u32x4_t* src[kLoads];
        int frag[kLoads], stride[kLoads];
#pragma unroll
        for (int i = 0; i < kLoads; ++i) {
            if (i < na) {
                const int j = na * wave + i;
                src[i] = wb + (size_t)tile_of(j >> 1) * ksteps * 64 + (j & 1) * 64 + lane;
                frag[i] = j;
                stride[i] = 128;
            } else {
                const int j = (kLoads - na) * wave + i - na;
                int n = 16 * (j >> 1) + r;
                n = n < ntok ? n : 0;          // padded token columns read a valid row; results dropped
                const int row = kGateUp ? ffn_token(p, xs, row0 + n) : row0 + n;
                const void* rows = kFp8 ? (kGateUp ? (const void*)p.xq : (const void*)p.hq) : (kGateUp ? p.x : p.h);
                src[i] = (const u32x4_t*)rows + (size_t)row * row_units + (j & 1) * 4 + g;
                frag[i] = bbase + j;
                stride[i] = 8;
            }
        }
        // Row scales, transposed and in permuted row order ([block][row]):
        // one 128-byte line per wave and block.
        const float* xsrc = nullptr;
        if (kFp8) {
            const int per = 1 << xsh;
            int n = per * wave + (lane & (per - 1));
            n = n < ntok ? n : 0;
            xsrc = (kGateUp ? p.xst : p.hst) + row0 + n;
        }
        auto issue = [&](int kb, GemmStage& s) __attribute__((always_inline)) {
#pragma unroll
            for (int i = 0; i < kLoads; ++i)
                __builtin_amdgcn_global_load_lds((const void*)(src[i] + (size_t)kb * stride[i]),
                                                 (lds_void_t*)&s.f[frag[i]][0], 16, 0, 0);
            if (kFp8)
                __builtin_amdgcn_global_load_lds((const void*)(xsrc + (size_t)kb * p.P), (lds_void_t*)&s.x[wave][0], 4,
                                                 0, 0);
        };
        // Weight tiles this wave multiplies: gate/up -> slots 2q, 2q+1 (gate)
        // and 4+2q, 5+2q (up); down -> slots 4q..4q+3.
        int aslot[4], srow[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            aslot[i] = kGateUp ? (i < 2 ? 2 * wq + i : kTiles / 2 + 2 * wq + i - 2) : 4 * wq + i;
            srow[i] = aslot[i] >= tiles / 2;
        }
        if (kFp8)
            for (int q = tid; q < 2 * kblocks; q += kGemmThreads) {
                const int h = q >= kblocks, kb = q - h * kblocks;
                const int row = (tile_of(h * (tiles / 2)) * 16) / 128;
                wsl[h][kb] = wsc[(size_t)row * kblocks + kb];
            }
        __syncthreads();

        f32x4_t acc[4][kWaveNT];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < kWaveNT; ++j) acc[i][j] = zero;

        // Multiplies block kb, held in stage s.
        auto compute = [&](int kb, const GemmStage& s) __attribute__((always_inline)) {
            if (!kFp8) {
                // bf16: the stage's two 64-byte steps are two MFMAs deep.
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    bf16x8_t af[4];
#pragma unroll
                    for (int i = 0; i < 4; ++i) af[i] = __builtin_bit_cast(bf16x8_t, s.f[2 * aslot[i] + h][lane]);
#pragma unroll
                    for (int j = 0; j < kWaveNT; ++j) {
                        const int n = kWaveNT * wc + j;
                        if (n < nb) {
                            const bf16x8_t bf = __builtin_bit_cast(bf16x8_t, s.f[bbase + 2 * n + h][lane]);
#pragma unroll
                            for (int i = 0; i < 4; ++i)
                                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bf, acc[i][j], 0, 0, 0);
                        }
                    }
                }
                return;
            }
            i32x8_t af[4];
            float ws[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                af[i] = join(s.f[2 * aslot[i]][lane], s.f[2 * aslot[i] + 1][lane]);
                ws[i] = wsl[srow[i]][kb];
            }
#pragma unroll
            for (int j = 0; j < kWaveNT; ++j) {
                const int n = kWaveNT * wc + j;
                if (n < nb) {
                    const i32x8_t bf = join(s.f[bbase + 2 * n][lane], s.f[bbase + 2 * n + 1][lane]);
                    const int tok = 16 * n + r;
                    const float xsv = s.x[tok >> xsh][tok & ((1 << xsh) - 1)];
                    f32x4_t part[4];
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        part[i] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(af[i], bf, zero, 0, 0, 0,
                                                                                  kScaleOne, 0, kScaleOne);
#pragma unroll
                    for (int i = 0; i < 4; ++i) acc[i][j] += part[i] * (ws[i] * xsv);
                }
            }
        };
        // Pipeline step v (< kblocks) issues block v into stage v % 3 and
        // multiplies block v - 2.  Before multiplying, the wave waits for its
        // own loads of block v - 2 (those of block v - 1 may stay in flight),
        // and a barrier makes every wave's loads visible; the same barrier
        // guarantees that all waves are done with block v - 3, whose stage
        // block v refills.  Waits and loads are unconditional and each stage
        // is named statically, so the compiler's wait analysis can tell that
        // the stage read is complete and adds no waits of its own.
        auto step = [&](int v, GemmStage& fill, const GemmStage& use) __attribute__((always_inline)) {
            wait_vm<kLoadsPerStage>();
            stage_barrier();
            issue(v, fill);
            if (v >= 2) compute(v - 2, use);
        };
        // The last two blocks, held in stages s2 (block kblocks - 2) and s1.
        auto tail = [&](const GemmStage& s2, const GemmStage& s1) __attribute__((always_inline)) {
            if (kblocks >= 2) {
                wait_vm<kLoadsPerStage>();
                stage_barrier();
                compute(kblocks - 2, s2);
            }
            wait_vm<0>();
            stage_barrier();
            compute(kblocks - 1, s1);
        };
        const int full = kblocks - kblocks % kStages;
#pragma clang loop unroll(disable)
        for (int v = 0; v < full; v += kStages) {
            step(v, st0, st1);
            step(v + 1, st1, st2);
            step(v + 2, st2, st0);
        }
        switch (kblocks % kStages) {
            case 0:
                tail(st1, st2);
                break;
            case 1:
                step(full, st0, st1);
                tail(st2, st0);
                break;
            default:
                step(full, st0, st1);
                step(full + 1, st1, st2);
                tail(st0, st1);
                break;
        }
        // All waves are done with the ring before the next item refills it.
        stage_barrier();
        if constexpr (kGateUp && kFp8 && kFuseQuant) {
            // Per token row: amax over the item's 128 SwiGLU values (this
            // lane's 8, the 4 lanes of the column, the row waves through
            // LDS), scale = amax / 448 (1 if zero), codes of value / scale:
            // the separate quantiser's arithmetic, so the codes are the same.
            float* red = reinterpret_cast<float*>(&st0);   // [wave][64 tokens]; the ring is idle
            float hv[kWaveNT][2][4];
#pragma unroll
            for (int j = 0; j < kWaveNT; ++j) {
                float m = 0.0f;
#pragma unroll
                for (int i = 0; i < 2; ++i)
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        hv[j][i][v] = silu_mul(acc[i][j][v], acc[i + 2][j][v]);
                        m = fmaxf(m, fabsf(hv[j][i][v]));
                    }
                m = fmaxf(m, __shfl_xor(m, 16));
                m = fmaxf(m, __shfl_xor(m, 32));
                if (g == 0) red[wave * 64 + 16 * j + r] = m;
            }
            __syncthreads();
#pragma unroll
            for (int j = 0; j < kWaveNT; ++j) {
                const int n = kWaveNT * wc + j, tn = 16 * n + r;
                float m = 0.0f;
#pragma unroll
                for (int q = 0; q < kRowWaves; ++q) m = fmaxf(m, red[(kRowWaves * wc + q) * 64 + 16 * j + r]);
                if (n >= nb || tn >= ntok) continue;
                const float sc = m > 0.0f ? m / kE4M3Max : 1.0f;
                const size_t row = (size_t)(row0 + tn);
#pragma unroll
                for (int i = 0; i < 2; ++i) {
                    const int col = (grp * (kTiles / 2) + 2 * wq + i) * 16 + 4 * g;
                    uint32_t word = 0;
#pragma unroll
                    for (int v = 0; v < 4; ++v) word |= e4m3_code(hv[j][i][v] / sc) << (8 * v);
                    *(uint32_t*)(p.hq + row * p.f + col) = word;
                }
                if (wq == 0 && g == 0) p.hst[(size_t)grp * p.P + row] = sc;
            }
            continue;
        }
#pragma unroll
        for (int j = 0; j < kWaveNT; ++j) {
            const int n = kWaveNT * wc + j, tn = 16 * n + r;
            if (n >= nb || tn >= ntok) continue;
            if (kGateUp) {
#pragma unroll
                for (int i = 0; i < 2; ++i) {
                    const int col = (grp * (kTiles / 2) + 2 * wq + i) * 16 + 4 * g;
                    float h[4];
#pragma unroll
                    for (int v = 0; v < 4; ++v) h[v] = silu_mul(acc[i][j][v], acc[i + 2][j][v]);
                    const size_t o = (size_t)(row0 + tn) * p.f + col;
                    if (kFp8) {
                        *(float4*)((float*)p.h + o) = make_float4(h[0], h[1], h[2], h[3]);
                    } else {   // bf16 SwiGLU rows, rounded to nearest even
                        uint2 pk;
                        pk.x = bf16_rne(h[0]) | (bf16_rne(h[1]) << 16);
                        pk.y = bf16_rne(h[2]) | (bf16_rne(h[3]) << 16);
                        *(uint2*)((uint16_t*)p.h + o) = pk;
                    }
                }
            } else {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    store_y4(p, (size_t)(row0 + tn), (grp * tiles + 4 * wq + i) * 16 + 4 * g, acc[i][j][0],
                             acc[i][j][1], acc[i][j][2], acc[i][j][3]);
                }
            }
        }
    }
}

// Block scales of x for the rows of the big chunks, transposed and in
// permuted row order: xst[b][row] = xs[token of row][b].  One workgroup per
// chunk, one thread per row (coalesced stores).
__global__ __launch_bounds__(256) void k_gather_xs(FfnParams p) {
    const int nblk = p.d / 128;
    for (int c = blockIdx.x; c < ffn_list_size(p); c += gridDim.x) {
        const ChunkRef ck = ffn_chunk(p, c);
        for (int n = threadIdx.x; n < ck.ntok; n += blockDim.x) {
            const int row = ck.row0 + n;
            const float* src = p.xs + (size_t)ffn_token(p, ck.xs, row) * nblk;
            for (int b = 0; b < nblk; ++b) p.xst[(size_t)b * p.P + row] = src[b];
        }
    }
}

}  // namespace

hipError_t launch_gather_xs(const FfnParams& p, int max_chunks, hipStream_t s) {
    const int blocks = max_chunks > 0 ? max_chunks : 1;
    hipLaunchKernelGGL(k_gather_xs, dim3((unsigned)blocks), dim3(256), 0, s, p);
    return hipGetLastError();
}

bool gemm_fp8_supports(const FfnParams& p, int nb) {
    return nb == kNT && p.tiled && p.f % 128 == 0 && p.d % 128 == 0 && p.d % (16 * kTiles) == 0 &&
           p.d / 128 <= kMaxKBlocks && p.f / 128 <= kMaxKBlocks;
}

bool gemm_fp8_applies(const caee_layer_desc_t& d, bool tiled) {
    return kGemmT > 0 && d.w_dtype == CAEE_FP8_E4M3 && d.T > kGemmT && tiled && d.f % 128 == 0 &&
           d.d % 128 == 0 && d.d % (16 * kTiles) == 0 && d.d / 128 <= kMaxKBlocks && d.f / 128 <= kMaxKBlocks;
}

int gemm_fp8_blocks() { return kNT; }

bool gemm_fp8_fuses_quant() { return kFuseQuant; }

// bf16: 64-element stages; gate/up items of kTiles / 2 features, down items
// of kTiles row tiles.
bool gemm_bf16_supports(const FfnParams& p, int nb) {
    return kGemmBf16 && nb == kNT && p.tiled && p.d % 64 == 0 && p.f % 64 == 0 && p.f % (8 * kTiles) == 0 &&
           p.d % (16 * kTiles) == 0;
}

bool gemm_bf16_applies(const caee_layer_desc_t& d, bool tiled) {
    return kGemmBf16 && d.w_dtype == CAEE_BF16 && tiled && d.d % 64 == 0 && d.f % 64 == 0 &&
           d.f % (8 * kTiles) == 0 && d.d % (16 * kTiles) == 0;
}

hipError_t launch_gemm(const FfnParams& p, bool gate_up, bool fp8, int max_chunks, hipStream_t s) {
    const int groups = gate_up ? p.f / (16 * kTiles / 2) : p.d / (16 * kTiles);
    // One workgroup per CU at a time (the ring fills the LDS); with the plain
    // order, two per CU so that a CU whose items end early takes more.
    long long items = (long long)max_chunks * groups;
    const long long cap = (long long)device_cu_count() * (CAEE_GEMM_XCD ? 1 : 2);
    if (items > cap) items = cap;
    if (items < 1) items = 1;
    const dim3 grid((unsigned)items), block(kGemmThreads);
    if (fp8) {
        if (gate_up) ffn_launch(k_gemm<true, true>, grid, block, s, p);
        else ffn_launch(k_gemm<false, true>, grid, block, s, p);
    } else {
        if (gate_up) ffn_launch(k_gemm<true, false>, grid, block, s, p);
        else ffn_launch(k_gemm<false, false>, grid, block, s, p);
    }
    return hipGetLastError();
}

}  // namespace caee
