// Prefill-class 8-bit expert products for big chunks (up to 128 rows).
//
// A workgroup computes a 256-weight-row x 128-token tile of one chunk over
// the whole contraction, one 128-wide block (one scaled 16x16x128 MFMA deep)
// per pipeline stage.  Weights (tiled order: the 2 KB of one 16-row tile and
// one block are contiguous), the chunk's token rows and the rows' block
// scales go straight from global memory to LDS with the 16-byte (and 4-byte)
// direct-to-LDS loads of gfx950, three stages in a ring, so that two stages
// of loads are in flight while one is multiplied and no register holds
// staged data.  Every wave issues the same number of loads per stage, so a
// wave waits for its oldest stage with a constant vmcnt, and one barrier per
// stage makes all waves' loads of that stage visible.
//
//   gate/up: the tile is 8 features (gate and up rows of each); wave w owns
//            features 2w, 2w+1 -> fp32 SwiGLU rows;
//   down:    the tile is 256 rows of W2; wave w owns 4 row tiles -> fp32 Y rows.
#include "caee_internal.h"

namespace caee {
namespace {

typedef int i32x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void_t;

constexpr int kScaleOne = 127;        // E8M0 1.0: the MFMA's own block scales are unused
constexpr int kTiles = 16;            // 16-row weight tiles per workgroup tile
constexpr int kNT = 8;                // 16-token tiles per workgroup tile (128 tokens)
constexpr int kStages = 3;
constexpr int kLoadsPerStage = 13;    // per wave: 8 weight, 4 row, 1 scale loads
constexpr int kMaxKBlocks = 128;      // contraction up to 16384

struct GemmStage {
    u32x4_t a[kTiles][2][kWave];      // weight fragments: [tile][half of the block][lane]
    u32x4_t b[kNT][2][kWave];         // token-row fragments: [token tile][half][lane]
    float x[4][kWave];                // row scales: token n at [n / 32][n % 32]
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

template <bool kGateUp>
__global__ __launch_bounds__(kFfnThreads) void k_gemm_fp8(FfnParams p) {
    // The ring's stages are separate LDS objects (and the loop below names
    // each statically), so the compiler can tell a read of one stage from the
    // loads still filling the others and does not wait for those.
    __shared__ GemmStage st0, st1, st2;
    // Weight block scales of the item: the tile's first and second half of
    // weight rows each fall in one 128-row scale row.  Read from LDS in the
    // pipeline, as a global load there would make the wave drain its loads.
    __shared__ float wsl[2][kMaxKBlocks];
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    const int r = lane & 15, g = lane >> 4;
    const int K = kGateUp ? p.d : p.f;                 // contraction length
    const int kblocks = K / 128;
    const size_t ksteps = (size_t)K / 64;              // 64-byte steps per weight row
    const size_t row_units = (size_t)K / 16;           // 16-byte pieces per token row
    const int rows_out = kGateUp ? p.f : p.d;          // features (gate/up) or output rows (down)
    const int groups = kGateUp ? rows_out / (16 * kTiles / 2) : rows_out / (16 * kTiles);
    const int n_chunks = ffn_list_size(p);
    const int total = n_chunks * groups;
    const size_t expert_bytes = kGateUp ? (size_t)2 * p.f * p.d : (size_t)p.d * p.f;
    const size_t scales_per_expert = (size_t)((kGateUp ? 2 * p.f : p.d) / 128) * kblocks;
    for (int item = blockIdx.x; item < total; item += gridDim.x) {
        const int c = item / groups, grp = item - c * groups;
        const ChunkRef ck = ffn_chunk(p, c);
        const int xs = ck.xs, row0 = ck.row0, ntok = ck.ntok;
        if (ffn_skip(p, xs)) continue;   // uniform over the workgroup
        const int nb = (ntok + 15) >> 4;
        const u32x4_t* wb = (const u32x4_t*)ffn_weights(p, xs, kGateUp ? false : true, expert_bytes);
        const float* wsc = ffn_scales(p, xs, kGateUp ? false : true, scales_per_expert);
        // Expert-relative weight tile of workgroup tile slot i.
        auto tile_of = [&](int i) {
            if (kGateUp) return i < kTiles / 2 ? grp * (kTiles / 2) + i : p.f / 16 + grp * (kTiles / 2) + i - kTiles / 2;
            return grp * kTiles + i;
        };
        // This wave's loads: weight tiles 4w..4w+3 (both halves), row blocks
        // j = 4w..4w+3 (token tile j/2, half j%2), and scales of tokens
        // 32w..32w+31 (lanes 32..63 repeat them into padding).
        const u32x4_t* asrc[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) asrc[i] = wb + (size_t)tile_of(4 * wave + i) * ksteps * 64 + lane;
        const u32x4_t* bsrc[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int j = 4 * wave + i, tb = j >> 1;
            int n = 16 * tb + r;
            n = n < ntok ? n : 0;          // padded token columns read a valid row; results dropped
            const int row = kGateUp ? ffn_token(p, xs, row0 + n) : row0 + n;
            bsrc[i] = (const u32x4_t*)(kGateUp ? (const void*)p.xq : (const void*)p.hq) + (size_t)row * row_units +
                      (j & 1) * 4 + g;
        }
        const float* xsrc;
        {
            int n = 32 * wave + (lane & 31);
            n = n < ntok ? n : 0;
            const int row = kGateUp ? ffn_token(p, xs, row0 + n) : row0 + n;
            xsrc = (kGateUp ? p.xs : p.hs) + (size_t)row * kblocks;
        }
        auto issue = [&](int kb, GemmStage& s) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int h = 0; h < 2; ++h)
                    __builtin_amdgcn_global_load_lds((const void*)(asrc[i] + (size_t)(2 * kb + h) * 64),
                                                     (lds_void_t*)&s.a[4 * wave + i][h][0], 16, 0, 0);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int j = 4 * wave + i;
                __builtin_amdgcn_global_load_lds((const void*)(bsrc[i] + (size_t)kb * 8),
                                                 (lds_void_t*)&s.b[j >> 1][j & 1][0], 16, 0, 0);
            }
            __builtin_amdgcn_global_load_lds((const void*)(xsrc + kb), (lds_void_t*)&s.x[wave][0], 4, 0, 0);
        };
        // Fragments this wave multiplies: gate/up -> slots 2w, 2w+1 (gate)
        // and 8+2w, 9+2w (up); down -> slots 4w..4w+3.
        int aslot[4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
            aslot[i] = kGateUp ? (i < 2 ? 2 * wave + i : kTiles / 2 + 2 * wave + i - 2) : 4 * wave + i;
        int srow[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) srow[i] = aslot[i] >= kTiles / 2;
        for (int q = tid; q < 2 * kblocks; q += kFfnThreads) {
            const int h = q >= kblocks, kb = q - h * kblocks;
            const int row = (tile_of(h * (kTiles / 2)) * 16) / 128;
            wsl[h][kb] = wsc[(size_t)row * kblocks + kb];
        }
        __syncthreads();

        f32x4_t acc[4][kNT];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int n = 0; n < kNT; ++n) acc[i][n] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        const f32x4_t zero = {0.f, 0.f, 0.f, 0.f};

        // One pipeline step: wait for this wave's loads of stage kb (the
        // loads of stage kb + 1 may stay in flight), make every wave's loads
        // visible, refill the stage freed by step kb - 1 with block kb + 2,
        // then multiply stage kb.
        auto step = [&](int kb, const GemmStage& s, GemmStage& ahead) {
            if (kb + 1 < kblocks) wait_vm<kLoadsPerStage>();
            else wait_vm<0>();
            stage_barrier();
            if (kb + 2 < kblocks) issue(kb + 2, ahead);
            i32x8_t af[4];
            float ws[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                af[i] = join(s.a[aslot[i]][0][lane], s.a[aslot[i]][1][lane]);
                ws[i] = wsl[srow[i]][kb];
            }
#pragma unroll
            for (int n = 0; n < kNT; ++n) {
                if (n < nb) {
                    const i32x8_t bf = join(s.b[n][0][lane], s.b[n][1][lane]);
                    const int tok = 16 * n + r;
                    const float xsv = s.x[tok >> 5][tok & 31];
                    f32x4_t part[4];
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        part[i] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(af[i], bf, zero, 0, 0, 0,
                                                                                  kScaleOne, 0, kScaleOne);
#pragma unroll
                    for (int i = 0; i < 4; ++i) acc[i][n] += part[i] * (ws[i] * xsv);
                }
            }
        };
        issue(0, st0);
        // Always a full second stage (block 0 again when there is one block;
        // never read), so that every path into the loop has the same loads
        // in flight and the compiler adds no wait of its own.
        issue(kblocks > 1 ? 1 : 0, st1);
        for (int kb = 0; kb < kblocks; kb += kStages) {
            step(kb, st0, st2);
            if (kb + 1 < kblocks) step(kb + 1, st1, st0);
            if (kb + 2 < kblocks) step(kb + 2, st2, st1);
        }
        // All waves are done with the ring before the next item refills it.
        stage_barrier();
#pragma unroll
        for (int n = 0; n < kNT; ++n) {
            const int tn = 16 * n + r;
            if (n >= nb || tn >= ntok) continue;
            if (kGateUp) {
#pragma unroll
                for (int i = 0; i < 2; ++i) {
                    const int col = (grp * (kTiles / 2) + 2 * wave + i) * 16 + 4 * g;
                    float h[4];
#pragma unroll
                    for (int v = 0; v < 4; ++v) h[v] = silu_mul(acc[i][n][v], acc[i + 2][n][v]);
                    *(float4*)((float*)p.h + (size_t)(row0 + tn) * p.f + col) = make_float4(h[0], h[1], h[2], h[3]);
                }
            } else {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    float* o = p.yperm + (size_t)(row0 + tn) * p.d + (grp * kTiles + 4 * wave + i) * 16 + 4 * g;
                    *(float4*)o = make_float4(acc[i][n][0], acc[i][n][1], acc[i][n][2], acc[i][n][3]);
                }
            }
        }
    }
}

}  // namespace

bool gemm_fp8_supports(const FfnParams& p, int nb) {
    return nb == kNT && p.tiled && p.f % 128 == 0 && p.d % 256 == 0 && p.d / 128 <= kMaxKBlocks &&
           p.f / 128 <= kMaxKBlocks;
}

hipError_t launch_gemm_fp8(const FfnParams& p, bool gate_up, int max_chunks, hipStream_t s) {
    const int groups = gate_up ? p.f / 128 : p.d / 256;
    long long items = (long long)max_chunks * groups;
    const long long cap = (long long)device_cu_count() * 2;
    if (items > cap) items = cap;
    if (items < 1) items = 1;
    if (gate_up) hipLaunchKernelGGL(k_gemm_fp8<true>, dim3((unsigned)items), dim3(kFfnThreads), 0, s, p);
    else hipLaunchKernelGGL(k_gemm_fp8<false>, dim3((unsigned)items), dim3(kFfnThreads), 0, s, p);
    return hipGetLastError();
}

}  // namespace caee
