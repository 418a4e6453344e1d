// LDS-pipelined bf16 expert products for the big chunks of a decode batch
// (experts with more rows of the call than a small chunk holds).
//
// A workgroup of 8 waves computes a 256-weight-row x 128-token tile (or,
// built with CAEE_GEMM_TILES=8, 128 x 256) of one chunk over the whole
// contraction, 128 bytes of each row (two 16x16x32 bf16 MFMAs deep) per
// pipeline stage.  Weights (tiled order: the 2 KB of one 16-row tile and one
// stage are contiguous) and the chunk's token rows go straight from global
// memory to LDS with the 16-byte direct-to-LDS loads of gfx950, three stages
// in a ring, so that two stages of loads are in flight while one is
// multiplied and no register holds staged data.  Every wave issues the same
// number of loads per stage, so a wave waits for its oldest stage with a
// constant vmcnt, and one barrier per stage makes all waves' loads of that
// stage visible.
//
// Each wave owns 4 weight tiles x 4 token tiles (64 x 64 outputs); two waves
// share a SIMD.  With R = kTiles / 4 waves across the rows, wave w = R * c + q
// takes token tiles 4c .. 4c + 3 and
//   gate/up: features 2q, 2q + 1 of the tile's kTiles / 2 (gate and up rows
//            of each) -> bf16 SwiGLU rows;
//   down:    row tiles 4q .. 4q + 3 -> fp32 expert output rows.
// (The 8-bit products of prefill batches run the register-weight kernel of
// ffn_prefill8.hip.)
#include "caee_internal.h"

namespace caee {
namespace {

typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void_t;
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));

// Workgroup tile: kTiles 16-row weight tiles x kNT 16-token tiles, 8 waves
// of 4 x 4 tiles each.
#ifndef CAEE_GEMM_TILES
#define CAEE_GEMM_TILES 16
#endif
constexpr int kTiles = CAEE_GEMM_TILES;
constexpr int kNT = 128 / kTiles;
constexpr int kWaveNT = 4;            // token tiles per wave
static_assert(kTiles == 8 || kTiles == 16, "tile shape");
// Whether the items are laid out by XCD (see the kernel; measured slower for
// these chunks, so off by default).
#ifndef CAEE_GEMM_XCD
#define CAEE_GEMM_XCD 0
#endif
constexpr int kStages = 3;
constexpr int kGemmWaves = 8;
constexpr int kGemmThreads = kGemmWaves * kWave;
// Fragments of one stage: 2 halves of every weight tile, then of every token
// tile.
constexpr int kFrags = 2 * (kTiles + kNT);
constexpr int kLoads = kTiles / 4 + kNT / 4;   // fragment loads per wave and stage
constexpr int kXcds = 8;              // accelerator complex dies, each with its own L2

// One stage: [2 * tile + half] the weight fragments (lane order), then the
// token rows' 128-byte blocks, row t at f[2 * kTiles + t / 8][8 (t % 8) ..],
// its 16-byte piece c in position c ^ (t % 8) (an XOR swizzle: the 8 lanes of
// a fragment read that take one piece each of 8 consecutive rows hit 8
// different bank groups; each row load brings 8 whole blocks).
struct GemmStage {
    u32x4_t f[kFrags][kWave];
};

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

template <bool kGateUp>
__global__ __launch_bounds__(kGemmThreads) void k_gemm(FfnParams p) {
    // The ring's stages are separate LDS objects (and the code below names
    // each statically), so the compiler can tell a read of one stage from the
    // loads still filling the others and does not wait for those.
    __shared__ GemmStage st0, st1, st2;
    const int tid = threadIdx.x, lane = tid & (kWave - 1);
    // Wave index as a scalar: the tile and fragment indices derived from it
    // stay in scalar registers.
    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
    const int r = lane & 15, g = lane >> 4;
    const int K = kGateUp ? p.d : p.f;                 // contraction length
    const int kblocks = K * 2 / 128;                   // pipeline stages (128 bytes of each row)
    const size_t ksteps = (size_t)K * 2 / 64;          // 64-byte steps per weight row
    const size_t row_units = (size_t)K * 2 / 16;       // 16-byte pieces per token row
    const int rows_out = kGateUp ? p.f : p.d;          // features (gate/up) or output rows (down)
    const int groups = kGateUp ? rows_out / (16 * kTiles / 2) : rows_out / (16 * kTiles);
    const int n_chunks = ffn_list_size(p);
    const int total = n_chunks * groups;
    const size_t expert_bytes = (kGateUp ? (size_t)2 * p.f * p.d : (size_t)p.d * p.f) * 2;
    const f32x4_t zero = {0.f, 0.f, 0.f, 0.f};
    constexpr int rw = kTiles / 4;                     // waves across the weight rows
    const int wq = wave % rw, wc = wave / rw;          // this wave's weight-row and token-column group
    constexpr int na = kTiles / 4;                     // weight fragment loads per wave (the rest: rows)
    constexpr int bbase = 2 * kTiles;                  // first token-row fragment of a stage
    // Workgroups go to the XCDs round robin (workgroup b to XCD b % 8).  With
    // a grid that is a multiple of 8, XCD x takes the x-th eighth of the item
    // list, so the items of one chunk (same token rows, different weight
    // groups) run at the same time on one XCD and share its L2.
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
        const int row0 = ck.row0, ntok = ck.ntok, grp = item - c * groups;
        const int nb = (ntok + 15) >> 4;
        const u32x4_t* wb = (const u32x4_t*)ffn_weights(p, xs, !kGateUp, expert_bytes);
        // Expert-relative weight tile of workgroup tile slot i.
        auto tile_of = [&](int i) {
            if (kGateUp) return i < kTiles / 2 ? grp * (kTiles / 2) + i : p.f / 16 + grp * (kTiles / 2) + i - kTiles / 2;
            return grp * kTiles + i;
        };
        // This wave's kLoads fragment loads per stage: (tile, half) pairs
        // j = na * w + i of the weights, then (token tile, half) pairs
        // j = (kLoads - na) * w + i of the rows.
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
                // Load j of the rows: 8 whole 128-byte blocks, lane l taking
                // piece (l % 8) ^ (l / 8) of row 8j + l / 8 (see GemmStage).
                const int j = (kLoads - na) * wave + i - na;
                int n = 8 * j + (lane >> 3);
                n = n < ntok ? n : 0;          // padded token columns read a valid row; results dropped
                const int row = kGateUp ? ffn_token(p, xs, row0 + n) : row0 + n;
                src[i] = (const u32x4_t*)(kGateUp ? p.x : p.h) + (size_t)row * row_units + ((lane & 7) ^ (lane >> 3));
                frag[i] = bbase + j;
                stride[i] = 8;
            }
        }
        auto issue = [&](int kb, GemmStage& s) __attribute__((always_inline)) {
#pragma unroll
            for (int i = 0; i < kLoads; ++i)
                __builtin_amdgcn_global_load_lds((const void*)(src[i] + (size_t)kb * stride[i]),
                                                 (lds_void_t*)&s.f[frag[i]][0], 16, 0, 0);
        };
        // Weight tiles this wave multiplies: gate/up -> slots 2q, 2q+1 (gate)
        // and kTiles/2 + 2q, kTiles/2 + 2q + 1 (up); down -> slots 4q..4q+3.
        int aslot[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) aslot[i] = kGateUp ? (i < 2 ? 2 * wq + i : kTiles / 2 + 2 * wq + i - 2) : 4 * wq + i;

        f32x4_t acc[4][kWaveNT];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < kWaveNT; ++j) acc[i][j] = zero;

        // This lane's B fragment of token tile n, half h: token 16n + r,
        // piece 4h + g of its block, at f[bbase + 2n] + fo[h].
        const int fo[2] = {(r >> 3) * kWave + (r & 7) * 8 + (g ^ (r & 7)),
                           (r >> 3) * kWave + (r & 7) * 8 + ((4 + g) ^ (r & 7))};
        // Multiplies the stage's two 64-byte steps, two MFMAs deep.
        auto compute = [&](const GemmStage& s) __attribute__((always_inline)) {
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                bf16x8_t af[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) af[i] = __builtin_bit_cast(bf16x8_t, s.f[2 * aslot[i] + h][lane]);
#pragma unroll
                for (int j = 0; j < kWaveNT; ++j) {
                    const int n = kWaveNT * wc + j;
                    if (n < nb) {
                        const bf16x8_t bf = __builtin_bit_cast(bf16x8_t, (&s.f[bbase + 2 * n][0])[fo[h]]);
#pragma unroll
                        for (int i = 0; i < 4; ++i)
                            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bf, acc[i][j], 0, 0, 0);
                    }
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
            wait_vm<kLoads>();
            stage_barrier();
            issue(v, fill);
            if (v >= 2) compute(use);
        };
        // The last two blocks, held in stages s2 (block kblocks - 2) and s1.
        auto tail = [&](const GemmStage& s2, const GemmStage& s1) __attribute__((always_inline)) {
            if (kblocks >= 2) {
                wait_vm<kLoads>();
                stage_barrier();
                compute(s2);
            }
            wait_vm<0>();
            stage_barrier();
            compute(s1);
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
                    // bf16 SwiGLU rows, rounded to nearest even
                    const size_t o = (size_t)(row0 + tn) * p.f + col;
                    uint2 pk;
                    pk.x = bf16_rne(h[0]) | (bf16_rne(h[1]) << 16);
                    pk.y = bf16_rne(h[2]) | (bf16_rne(h[3]) << 16);
                    *(uint2*)((uint16_t*)p.h + o) = pk;
                }
            } else {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    store_y4(p, (size_t)(row0 + tn), (grp * kTiles + 4 * wq + i) * 16 + 4 * g, acc[i][j][0],
                             acc[i][j][1], acc[i][j][2], acc[i][j][3]);
                }
            }
        }
    }
}

}  // namespace

int gemm_bf16_blocks() { return kNT; }

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

hipError_t launch_gemm(const FfnParams& p, bool gate_up, int max_chunks, hipStream_t s) {
    const int groups = gate_up ? p.f / (16 * kTiles / 2) : p.d / (16 * kTiles);
    // One workgroup per CU at a time (the ring fills most of the LDS); with
    // the plain order, two per CU so that a CU whose items end early takes more.
    long long items = (long long)max_chunks * groups;
    const long long cap = (long long)device_cu_count() * (CAEE_GEMM_XCD ? 1 : 2);
    if (items > cap) items = cap;
    if (items < 1) items = 1;
    const dim3 grid((unsigned)items), block(kGemmThreads);
    if (gate_up) ffn_launch(k_gemm<true>, grid, block, s, p);
    else ffn_launch(k_gemm<false>, grid, block, s, p);
    return hipGetLastError();
}

}  // namespace caee
