// 8-bit expert products of prefill batches: e4m3 weights (fp32 128x128
// block scales) against e4m3 token rows (fp32 scale per row and 128-wide
// block), for the big chunks of an 8-bit layer (experts with more rows than
// a small chunk, cut into near-equal chunks of at most 256 rows).
//
// A workgroup of 8 waves computes 256 weight rows x (up to) 256 tokens of
// one chunk over the whole contraction, one 128-deep block per pipeline
// stage:
//   * the chunk's token rows (and their block scales) go global -> LDS with
//     direct-to-LDS buffer loads, each load 8 whole 128-byte row blocks
//     (16 half rows per load measured 5 % slower), three stages ahead of
//     their multiply in a ring of four, issued among the multiplies of the
//     stage before; every wave reads every token fragment of a stage from
//     LDS;
//   * each wave owns two 16-row weight tiles (32 rows), which nobody else
//     reads: they go global -> registers, three stages ahead of their MFMAs
//     (two for items of more than 12 token tiles, whose accumulators leave
//     room for three register sets only), issued before the stage's wait,
//     and never pass through LDS.
// So a chunk of up to 256 rows (every routed expert of a 4096-token batch of
// the DeepSeek-R1 layer) streams each of its weight bytes once, and the
// bytes in flight per CU are the token ring's plus every wave's register
// stages.  An item is compiled for its chunk's token-tile count (1 .. 16),
// so every stage is straight-line code:
// per stage a wave issues the same loads (four weight pieces, its share of
// the token fragments, one row-scale load) and waits for its oldest stage
// with a constant vmcnt, one barrier per stage publishes the ring's stage to
// all waves, and the multiplies of a stage are software-pipelined over the
// token tiles (fragment reads two tiles ahead, scaling one tile behind).
//
// Work items: (chunk, run of weight groups); gate/up groups are 128 features
// (the gate and up rows of each; wave w takes feature tile w of both), down
// groups 256 output rows (wave w takes tiles 2w, 2w + 1).  An item runs its
// groups one after another through one pipeline.  Each gate/up group ends in
// SwiGLU and quantises its 128 features per token (amax across the waves
// through LDS) into e4m3 codes and a transposed block scale, the input of
// the down product; each down group writes bf16 expert output rows.
//
// Per block: one scaled 16x16x128 MFMA (unit E8M0 scales) per (weight tile,
// token tile), its partial sums times weight block scale x row block scale
// added in fp32.
#include "caee_internal.h"
#include "fp8_codec.h"

#include <type_traits>

namespace caee {
namespace {

typedef int i32x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void_t;
typedef const __attribute__((address_space(1))) u32x4_t g_u32x4_t;

constexpr int kP8Waves = 8;
constexpr int kP8Threads = kP8Waves * kWave;
// Token tiles of an item at most (16 tokens each: chunks of up to 256 rows).
constexpr int kP8NT = 16;
constexpr int kP8MaxKBlocks = 128;        // contraction up to 16384
constexpr int kBufWord3 = 0x00020000;      // buffer descriptor word 3: 32-bit data format, raw access
constexpr int kScaleOne = 127;            // E8M0 1.0: the MFMA's own block scales are unused
constexpr int kXcds = 8;                  // accelerator complex dies, each with its own L2
// Items grouped by XCD: all weight groups of a chunk run on one XCD, so its
// token rows are fetched into one L2 once (workgroups go to the XCDs round
// robin, workgroup b to XCD b % 8).
#ifndef CAEE_P8_XCD
#define CAEE_P8_XCD 1
#endif

// One stage of the token ring: the chunk's rows' 128-byte blocks, row t at
// f[t / 8][8 (t % 8) ..]: its 16-byte piece c in position c ^ (t % 8) (an
// XOR swizzle, so that the 8 lanes of a fragment read that take one piece
// each of 8 consecutive rows hit 8 different bank groups).
struct P8Stage {
    u32x4_t f[2 * kP8NT][kWave];
    float x[kP8Waves][kWave];             // row block scales: token n at [n / 32][n % 32]
};

__device__ inline i32x8_t join(const u32x4_t& lo, const u32x4_t& hi) {
    return i32x8_t{(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3], (int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
}

// silu(g) * u with the hardware reciprocal (about one ulp; the quantiser
// that follows rounds to 3 mantissa bits).
__device__ inline float silu_mul(float g, float u) { return g * __builtin_amdgcn_rcpf(1.0f + __expf(-g)) * u; }

// Waits until at most N of this wave's vector memory loads are outstanding
// (gfx9 s_waitcnt: vmcnt in bits 3:0 and 15:14, expcnt and lgkmcnt not waited).
template <int N>
__device__ inline void wait_vm() {
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | (((N >> 4) & 3) << 14));
}

// Waits until this wave's LDS (and scalar memory) operations are done.
__device__ inline void wait_lgkm0() { __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14)); }

// Workgroup barrier without the memory fence of __syncthreads (which would
// wait for every load in flight); the empty asm keeps the compiler from
// moving memory accesses across it.
__device__ inline void stage_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// Weight pieces of one stage in registers: [tile][half].
struct WReg {
    u32x4_t v[2][2];
};

template <int N>
using IntC = std::integral_constant<int, N>;

// f(IntC<B>{}), ..., f(IntC<E - 1>{}): a loop whose index is a constant in
// every copy of the body.
template <int B, int E, class F>
__device__ __attribute__((always_inline)) inline void static_for(F&& f) {
    if constexpr (B < E) {
        f(IntC<B>{});
        static_for<B + 1, E>(f);
    }
}

// Token tiles whose fragments a stage's multiply reads from LDS ahead of
// their MFMAs: two, or one for the widest items (whose accumulators leave no
// registers for a third fragment).
#ifndef CAEE_P8_AHEAD_MAX_NB
#define CAEE_P8_AHEAD_MAX_NB 12
#endif
constexpr int kP8Ahead(int nb) { return nb <= CAEE_P8_AHEAD_MAX_NB ? 2 : 1; }

// Weight register sets of a stage loop: four (weights loaded three blocks
// ahead of their multiply) up to this many token tiles, three (two blocks
// ahead) above, where the accumulators leave no room for a fourth set.
#ifndef CAEE_P8_W4_MAX_NB
#define CAEE_P8_W4_MAX_NB 12
#endif
constexpr int kP8WSets(int nb) { return nb <= CAEE_P8_W4_MAX_NB ? 4 : 3; }

// Weight groups an item runs back to back over its chunk (gate/up, down).
// The token ring and the weight stream carry on from one group into the
// next, so only the item's first group waits for a filling pipeline, and a
// group's epilogue runs while the next group's first blocks are in flight.
// Contractions that are not a multiple of four blocks run one group per item.
// Down (16-block contraction at d = 7168, f = 2048: short items) runs four;
// gate/up one: with fewer items per chunk more chunks are in flight per XCD
// and their token rows (7 KB each) no longer fit its L2 together (two groups:
// gate/up 7 % slower; down with seven groups per item: uneven tail).
#ifndef CAEE_P8_RUN_GU
#define CAEE_P8_RUN_GU 1
#endif
#ifndef CAEE_P8_RUN_DN
#define CAEE_P8_RUN_DN 4
#endif
constexpr int kP8MaxRun = 8;
// Widest items (token tiles) whose groups run back to back; wider ones run
// their groups one pipeline each (their accumulators leave no registers for
// a group epilogue inside the stage loop).
#ifndef CAEE_P8_RUN_MAX_NB
#define CAEE_P8_RUN_MAX_NB 12
#endif
static_assert(CAEE_P8_RUN_GU >= 1 && CAEE_P8_RUN_GU <= kP8MaxRun && CAEE_P8_RUN_DN >= 1 &&
                  CAEE_P8_RUN_DN <= kP8MaxRun,
              "groups per item");

// Token-row loads of a step issued among the multiplies of its tiles (1), or
// all at once before them (0).  (Spreading the weight loads the same way
// measured slower.)
#ifndef CAEE_P8_SPREAD
#define CAEE_P8_SPREAD 1
#endif

// Workgroups of the launch per CU (one runs at a time: the ring takes most
// of the LDS).
#ifndef CAEE_P8_GRID_PER_CU
#define CAEE_P8_GRID_PER_CU 2
#endif

// Token tiles an item is compiled for: its chunk's count rounded up to an
// even number (1), or the count itself (0).
#ifndef CAEE_P8_EVEN
#define CAEE_P8_EVEN 0
#endif

template <bool kGateUp>
__global__ __launch_bounds__(kP8Threads) void k_prefill8(FfnParams p) {
#if defined(__HIP_DEVICE_COMPILE__)   // the buffer-descriptor type exists for the GPU target only
    // Token ring: block v's token fragments and row scales in slot v % 4.
    // Four LDS objects, each named statically below, so that the compiler
    // can tell a read of one slot from the loads filling another.
    __shared__ P8Stage st0, st1, st2, st3;
    // Weight block scales of the item's groups: group q's two 128-row scale
    // rows at wsl[2q], wsl[2q + 1].
    constexpr int kRun = kGateUp ? CAEE_P8_RUN_GU : CAEE_P8_RUN_DN;
    __shared__ float wsl[2 * kRun][kP8MaxKBlocks];
    // Per-token maxima of the gate/up epilogue, [wave][token].
    __shared__ float red[kGateUp ? kP8Waves * 256 : 1];
    const int tid = threadIdx.x, lane = tid & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
    const int r = lane & 15, g = lane >> 4;
    const int K = kGateUp ? p.d : p.f;
    const int kblocks = K / 128;
    const size_t ksteps = (size_t)K / 64;          // 64-byte steps of a weight row (tiled layout)
    const size_t row_units = (size_t)K / 16;       // 16-byte pieces of a token row
    const int groups = kGateUp ? p.f / 128 : p.d / 256;
    // Groups per item (uniform): a run of up to G groups of one chunk.
    const int G = kblocks % 4 == 0 ? kRun : 1;
    const int runs = (groups + G - 1) / G;
    const int total = ffn_list_size(p) * runs;
    // Weight tiles from one group to the next (gate/up: 8 feature tiles of
    // the gate rows and of the up rows; down: 16 row tiles), in 16-byte units
    // (a run of groups spans less than 2^32 of them: K < 2^16).
    const uint32_t gstride = (uint32_t)(kGateUp ? 8 : 16) * (uint32_t)ksteps * 64u;
    const size_t expert_bytes = kGateUp ? (size_t)2 * p.f * p.d : (size_t)p.d * p.f;
    const size_t scales_per_expert = (size_t)((kGateUp ? 2 * p.f : p.d) / 128) * kblocks;
    const f32x4_t zero = {0.f, 0.f, 0.f, 0.f};
    // Token rows (e4m3 codes) and their transposed block scales; loads past
    // the end of a buffer return zero.
    const uint32_t tbytes = kGateUp ? (uint32_t)((size_t)p.T * p.d) : (uint32_t)((size_t)p.P * p.f);
    const uint32_t sbytes = (uint32_t)((size_t)kblocks * p.P * 4);
    const __amdgpu_buffer_rsrc_t tbuf =
        __builtin_amdgcn_make_buffer_rsrc((void*)(kGateUp ? p.xq : p.hq), 0, (int)tbytes, kBufWord3);
    const __amdgpu_buffer_rsrc_t sbuf =
        __builtin_amdgcn_make_buffer_rsrc((void*)(kGateUp ? p.xst : p.hst), 0, (int)sbytes, kBufWord3);

    // Item order: plain (workgroup b takes items b, b + grid, ...), or by
    // XCD (XCD x takes the chunks x, x + 8, ..., all group runs of each, its
    // workgroups striding through that list).
    const bool by_xcd = CAEE_P8_XCD && gridDim.x % kXcds == 0;
    const int xcd = blockIdx.x % kXcds;
    const int n_local = by_xcd ? (ffn_list_size(p) - xcd + kXcds - 1) / kXcds * runs : total;
    for (int it = by_xcd ? blockIdx.x / kXcds : blockIdx.x; it < n_local;
         it += by_xcd ? gridDim.x / kXcds : gridDim.x) {
        const int c = by_xcd ? xcd + kXcds * (it / runs) : it / runs;
        const int g0 = (it % runs) * G;                 // the item's first group
        const int gn = groups - g0 < G ? groups - g0 : G;
        const ChunkRef ck = ffn_chunk(p, c);
        const int xs = ck.xs;
        if (ffn_skip(p, xs)) continue;   // uniform over the workgroup
        const int row0 = ck.row0, ntok = ck.ntok;
        const int nb = (ntok + 15) >> 4;
        const u32x4_t* wb = (const u32x4_t*)ffn_weights(p, xs, !kGateUp, expert_bytes);
        const float* wsc = ffn_scales(p, xs, !kGateUp, scales_per_expert);
        // This wave's weight tiles in the first group (group q's are gstride
        // further) and which of a group's two scale rows they fall in.
        const int t0 = kGateUp ? g0 * 8 + wave : g0 * 16 + 2 * wave;
        const int t1 = kGateUp ? p.f / 16 + g0 * 8 + wave : t0 + 1;
        const int ws0 = kGateUp ? 0 : (wave >= 4 ? 1 : 0), ws1 = kGateUp ? 1 : ws0;
        const u32x4_t* wsrc[2] = {wb + (size_t)t0 * ksteps * 64 + lane, wb + (size_t)t1 * ksteps * 64 + lane};
        // Row scales, transposed and in permuted row order ([block][row]):
        // wave w loads tokens 32w .. 32w + 31 (lanes 32..63 repeat them).
        int xn = 32 * wave + (lane & 31);
        xn = xn < ntok ? xn : 0;
        // Byte offsets within the buffers the direct-to-LDS loads read (the
        // host keeps every buffer below 4 GiB): buffer loads, whose waits the
        // compiler counts apart from the LDS reads of the multiply.
        const uint32_t xoff = (uint32_t)(row0 + xn) * 4u;

        for (int q = tid; q < 2 * gn * kblocks; q += kP8Threads) {
            const int h = q / kblocks, kb = q - h * kblocks;   // group h / 2, its scale row h % 2
            const int gq = g0 + (h >> 1);
            const int srow = kGateUp ? ((h & 1) ? p.f / 128 + gq : gq) : 2 * gq + (h & 1);
            wsl[h][kb] = wsc[(size_t)srow * kblocks + kb];
        }
        __syncthreads();

        // The item for NB token tiles (the chunk's tile count, or that count
        // rounded up to an even number): loads, multiplies and waits are all
        // fixed by NB, so each stage is straight-line code whose waits the
        // compiler can count exactly.
        auto run = [&](auto nbc) __attribute__((always_inline)) {
            constexpr int NB = decltype(nbc)::value;
            // Token loads of a stage: 2 NB of 8 rows each, kTok per wave;
            // loads past 2 NB (when 8 kTok > 2 NB) read row 0 into stage
            // slots nobody multiplies.
            constexpr int kTok = (2 * NB + kP8Waves - 1) / kP8Waves;
            constexpr int kLoads = kTok + 1 + 4;   // + row scales + two tiles x two halves of weights
            static_assert(kTok * kP8Waves <= 2 * kP8NT, "stage slots");
            uint32_t toff[kTok];
#pragma unroll
            for (int i = 0; i < kTok; ++i) {
                const int j = kTok * wave + i;
                int n = 8 * j + (lane >> 3);   // lane l: piece (l % 8) ^ (l / 8) of row 8j + l / 8
                n = n < ntok ? n : 0;          // padded token columns read a valid row; results dropped
                const uint32_t row = kGateUp ? (uint32_t)ffn_token(p, xs, row0 + n) : (uint32_t)(row0 + n);
                toff[i] = (row * (uint32_t)row_units + (uint32_t)((lane & 7) ^ (lane >> 3))) * 16u;
            }
            // This lane's B fragment of token tile n: token 16n + r, pieces g
            // and 4 + g of its block, at f[2n] + these offsets (16-byte units).
            const int fo0 = (r >> 3) * kWave + (r & 7) * 8 + (g ^ (r & 7));
            const int fo1 = (r >> 3) * kWave + (r & 7) * 8 + ((4 + g) ^ (r & 7));

            auto issue_tok = [&](int kb, P8Stage& s) __attribute__((always_inline)) {
#pragma unroll
                for (int i = 0; i < kTok; ++i)
                    __builtin_amdgcn_raw_ptr_buffer_load_lds(tbuf, (lds_void_t*)&s.f[kTok * wave + i][0], 16, toff[i],
                                                             kb * 128, 0, 0);
                __builtin_amdgcn_raw_ptr_buffer_load_lds(sbuf, (lds_void_t*)&s.x[wave][0], 4, xoff, kb * p.P * 4, 0, 0);
            };
            // Weights of a block at offset wo (16-byte units) from each tile's start.
            auto issue_w = [&](uint32_t wo, WReg& w) __attribute__((always_inline)) {
#pragma unroll
                for (int t = 0; t < 2; ++t)
#pragma unroll
                    for (int h = 0; h < 2; ++h)
                        w.v[t][h] = __builtin_nontemporal_load((g_u32x4_t*)(wsrc[t] + (wo + (uint32_t)h * 64u)));
            };

            f32x4_t acc[2][NB];

            // One stage: per token tile two MFMAs (one per weight tile) on its
            // fragment.  Software-pipelined over the tiles: while tile n's
            // MFMAs run, the fragment and row scale of tile n + 2 are read
            // from LDS and tile n - 1's partial sums (its MFMAs are done) are
            // scaled into their accumulators, so neither the LDS latency nor
            // the MFMA latency is waited for in line.
            // Load k of a step (kTok token fragments, the row scales, then the
            // four weight pieces): compute() can spread the token loads over
            // its tiles.
            auto issue_one = [&](auto kc, int vt, P8Stage& st, uint32_t vw, WReg& w) __attribute__((always_inline)) {
                constexpr int k = decltype(kc)::value;
                if constexpr (k < kTok) {
                    __builtin_amdgcn_raw_ptr_buffer_load_lds(tbuf, (lds_void_t*)&st.f[kTok * wave + k][0], 16, toff[k],
                                                             vt * 128, 0, 0);
                } else if constexpr (k == kTok) {
                    __builtin_amdgcn_raw_ptr_buffer_load_lds(sbuf, (lds_void_t*)&st.x[wave][0], 4, xoff, vt * p.P * 4, 0,
                                                             0);
                } else {
                    constexpr int q = k - kTok - 1, t = q >> 1, h = q & 1;
                    w.v[t][h] = __builtin_nontemporal_load((g_u32x4_t*)(wsrc[t] + (vw + (uint32_t)h * 64u)));
                }
            };
            auto compute = [&](int q, int kb, const P8Stage& s, const WReg& w, int vt, P8Stage& st, uint32_t vw,
                               WReg& wn) __attribute__((always_inline)) {
                const i32x8_t a0 = join(w.v[0][0], w.v[0][1]), a1 = join(w.v[1][0], w.v[1][1]);
                const float wa = wsl[2 * q + ws0][kb], wc = wsl[2 * q + ws1][kb];
                auto frag = [&](int n) __attribute__((always_inline)) {
                    const u32x4_t* b = &s.f[2 * n][0];
                    return join(b[fo0], b[fo1]);
                };
                auto xsc = [&](int n) __attribute__((always_inline)) {
                    const int tok = 16 * n + r;
                    return s.x[tok >> 5][tok & 31];
                };
                constexpr int D = kP8Ahead(NB);   // fragment reads ahead of their MFMAs
                i32x8_t bq[D + 1];
                float xq[D + 1];
#pragma unroll
                for (int n = 0; n < D && n < NB; ++n) {
                    bq[n] = frag(n);
                    xq[n] = xsc(n);
                }
                f32x4_t pp0 = zero, pp1 = zero;
                float ps0 = 0.0f, ps1 = 0.0f;
                static_for<0, NB>([&](auto nc) __attribute__((always_inline)) {
                    constexpr int n = decltype(nc)::value;
                    if constexpr (n + D < NB) {
                        bq[(n + D) % (D + 1)] = frag(n + D);
                        xq[(n + D) % (D + 1)] = xsc(n + D);
                    }
                    const i32x8_t& b = bq[n % (D + 1)];
                    const f32x4_t q0 =
                        __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a0, b, zero, 0, 0, 0, kScaleOne, 0, kScaleOne);
                    const f32x4_t q1 =
                        __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a1, b, zero, 0, 0, 0, kScaleOne, 0, kScaleOne);
                    if constexpr (n > 0) {
                        acc[0][n - 1] += pp0 * ps0;
                        acc[1][n - 1] += pp1 * ps1;
                    }
                    pp0 = q0;
                    pp1 = q1;
                    ps0 = wa * xq[n % (D + 1)];
                    ps1 = wc * xq[n % (D + 1)];
                    // Issue order within the tile: its two MFMAs, the LDS
                    // reads of tile n + D, then the VALU work (tile n - 1's
                    // scaling, whose MFMAs are done by now, and tile n's
                    // scale factors).
                    // Token-row loads of this tile: [n L / NB, (n + 1) L / NB) of the
                    // step's L = kTok + 1.
                    constexpr int lo = CAEE_P8_SPREAD ? n * (kTok + 1) / NB : 0;
                    constexpr int hi = CAEE_P8_SPREAD ? (n + 1) * (kTok + 1) / NB : 0;
                    static_for<lo, hi>([&](auto kc) __attribute__((always_inline)) { issue_one(kc, vt, st, vw, wn); });
                    __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
                    static_for<lo, hi>([&](auto) __attribute__((always_inline)) {
                        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
                    });
                    if constexpr (n + D < NB) __builtin_amdgcn_sched_group_barrier(0x100, 3, 0);
                    if constexpr (n > 0) __builtin_amdgcn_sched_group_barrier(0x002, 10, 0);
                    else __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);
                    __builtin_amdgcn_sched_barrier(0);
                });
                acc[0][NB - 1] += pp0 * ps0;
                acc[1][NB - 1] += pp1 * ps1;
            };

            // Group outputs: the SwiGLU rows of group q (gate/up, quantised)
            // or its expert output rows (down) from the accumulators.
            auto epilogue = [&](int q) __attribute__((always_inline)) {
                if constexpr (kGateUp) {
                    // Lane (r, g) holds features 16 * wave + 4g .. + 3 of the
                    // group for token 16n + r.  Per token: amax over the
                    // group's 128 SwiGLU values (this lane's 4, the 4 lanes of
                    // the column, the 8 waves through LDS), scale = amax / 448
                    // (1 if zero), codes of value / scale: the activation
                    // quantiser's arithmetic.  The SwiGLU values replace the
                    // gate sums in place.
                    const int grp = g0 + q;
#pragma unroll
                    for (int n = 0; n < NB; ++n) {
                        float m = 0.0f;
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            acc[0][n][e] = silu_mul(acc[0][n][e], acc[1][n][e]);
                            m = fmaxf(m, fabsf(acc[0][n][e]));
                        }
                        m = fmaxf(m, __shfl_xor(m, 16));
                        m = fmaxf(m, __shfl_xor(m, 32));
                        if (g == 0) red[wave * 256 + 16 * n + r] = m;
                    }
                    // Every wave's maxima are in LDS (no wait for memory: the
                    // loads of the stages ahead and earlier stores stay in flight).
                    wait_lgkm0();
                    stage_barrier();
#pragma unroll
                    for (int n = 0; n < NB; ++n) {
                        int tn = 16 * n + r;
                        asm volatile("" : "+v"(tn));   // keeps the row arithmetic here, out of the stage loop
                        if (n >= nb || tn >= ntok) continue;
                        float m = 0.0f;
#pragma unroll
                        for (int w = 0; w < kP8Waves; ++w) m = fmaxf(m, red[w * 256 + tn]);
                        const float sc = m > 0.0f ? m / kE4M3Max : 1.0f;
                        const size_t row = (size_t)(row0 + tn);
                        const uint32_t word = e4m3_code4(acc[0][n][0] / sc, acc[0][n][1] / sc, acc[0][n][2] / sc,
                                                         acc[0][n][3] / sc);
                        *(uint32_t*)(p.hq + row * p.f + grp * 128 + 16 * wave + 4 * g) = word;
                        if (wave == 0 && g == 0) p.hst[(size_t)grp * p.P + row] = sc;
                    }
                } else {
#pragma unroll
                    for (int n = 0; n < NB; ++n) {
                        int tn = 16 * n + r;
                        asm volatile("" : "+v"(tn));   // keeps the row arithmetic here, out of the stage loop
                        if (n >= nb || tn >= ntok) continue;
#pragma unroll
                        for (int t = 0; t < 2; ++t)
                            store_y4(p, (size_t)(row0 + tn), (t ? t1 : t0) * 16 + 256 * q + 4 * g, acc[t][n][0],
                                     acc[t][n][1], acc[t][n][2], acc[t][n][3]);
                    }
                }
            };

            // One pipeline over groups qbase .. qbase + qn - 1 of the item: its
            // blocks u = 0 .. qn kblocks - 1 run group after group (block kb
            // of group qbase + q is u = q kblocks + kb), the token ring cycling
            // through the chunk's blocks once per group and the weights moving
            // on to the group's tiles.  Items wider than the chained limit run
            // one pipeline per group (qn = 1).
            constexpr bool kChain = kRun > 1 && NB <= CAEE_P8_RUN_MAX_NB;
            auto pipeline = [&](int qbase, int qn) __attribute__((always_inline)) {
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
                for (int n = 0; n < NB; ++n) acc[t][n] = zero;
            const int nblk = qn * kblocks;
            auto split = [&](int u, int& q, int& kb) __attribute__((always_inline)) {
                if constexpr (kChain) {
                    q = 0;
                    kb = u;
#pragma unroll
                    for (int i = 1; i < kRun; ++i)
                        if (kb >= kblocks) {
                            kb -= kblocks;
                            ++q;
                        }
                } else {
                    q = 0;
                    kb = u;
                }
                q += qbase;
            };

            // Token rows go three blocks ahead of their multiply (ring of
            // four), weights three (four register sets) or two (three sets):
            // step v issues the weights of block v + 1 (or v), then waits
            // until this wave's tokens and weights of block v - 2 have
            // landed (loads complete in order, so a constant count of later
            // loads may stay outstanding), passes a barrier that publishes
            // every wave's token loads of block v - 2 and guarantees that all
            // waves are done with block v - 3, whose ring slot the tokens of
            // block v + 1 then refill, and multiplies block v - 2.  Every step
            // issues the same loads (steps past the last block re-read it,
            // from L2, into a slot nobody multiplies), so the waits are
            // constants (a group epilogue's stores only make them stricter),
            // and the accumulators live in one set of registers throughout.
            constexpr int NW = kP8WSets(NB);
            WReg w0, w1, w2, w3;
            auto slot = [&](auto jc) -> P8Stage& {
                constexpr int J = decltype(jc)::value & 3;
                if constexpr (J == 0) return st0;
                else if constexpr (J == 1) return st1;
                else if constexpr (J == 2) return st2;
                else return st3;
            };
            auto wset = [&](auto jc) -> WReg& {
                constexpr int J = decltype(jc)::value % NW;
                if constexpr (J == 0) return w0;
                else if constexpr (J == 1) return w1;
                else if constexpr (J == 2) return w2;
                else return w3;
            };
            // Step v (J = v mod 12 static: slot and register set are named)
            // issues the loads of block v + 1 (tokens) and v + NW - 3
            // (weights) and, if kMult, multiplies block v - 2.  With four
            // sets it waits for the loads of step v - 3 (the tokens and
            // weights of block v - 2).
            auto step = [&](int v, auto jc, auto mc) __attribute__((always_inline)) {
                constexpr int J = decltype(jc)::value;
                constexpr bool kMult = decltype(mc)::value;
                // The weights first: their register set last held block
                // v - 3, which this wave multiplied in the previous step, so
                // they need no barrier and are in flight during the wait.
                const int uw = v + NW - 3 < nblk ? v + NW - 3 : nblk - 1;
                int qw, kw;
                split(uw, qw, kw);
                const uint32_t vw = (uint32_t)qw * gstride + (uint32_t)kw * 128u;   // this step's weight block
                issue_w(vw, wset(IntC<J + NW - 3>{}));
                // Block v - 2's tokens and weights have landed once at most
                // the loads issued after its weights are outstanding: its
                // tokens, the next steps' loads and these weights.
                if constexpr (NW == 4) wait_vm<2 * kLoads + 4>();
                else wait_vm<2 * kLoads>();
                stage_barrier();
                // A group other than the item's last ended with the previous
                // step's multiply (block v - 3): its outputs leave the
                // accumulators here, before this step's loads, while the
                // loads of the next blocks are in flight.  (With kblocks a
                // multiple of four that step is always v = 4 m + 2.)
                if constexpr (kChain && kMult && (J & 3) == 2) {
                    const int ub = v - 2;
                    int qe, ke;
                    split(ub, qe, ke);
                    if (ke == 0 && qe > qbase) {
                        epilogue(qe - 1);
#pragma unroll
                        for (int t = 0; t < 2; ++t)
#pragma unroll
                            for (int n = 0; n < NB; ++n) acc[t][n] = zero;
                    }
                }
                const int ut = v + 1 < nblk ? v + 1 : nblk - 1;
                int qt, vt;
                split(ut, qt, vt);
                (void)qt;
                // Steps without a multiply issue their token loads here, the
                // others inside compute().
                if constexpr (!kMult || !CAEE_P8_SPREAD) issue_tok(vt, slot(IntC<J + 1>{}));
                if constexpr (kMult) {
                    int qm, km;
                    split(v - 2, qm, km);
                    compute(qm, km, slot(IntC<J + 2>{}), wset(IntC<J + NW - 2>{}), vt, slot(IntC<J + 1>{}), vw,
                            wset(IntC<J + NW - 3>{}));
                }
            };
            // Steps 0 and 1 only load; steps 2 .. nblk + 1 multiply blocks
            // 0 .. nblk - 1: a loop over whole bodies of L steps (the lcm of
            // the ring and the register sets), then the remaining steps one
            // after another.  The loop body has a single path, so the
            // compiler's count of the loads between a register load and its
            // use is the real one and it adds no waits of its own.
            constexpr int L = NW == 4 ? 4 : 12;
            const int vend = nblk + 2;
            issue_tok(0, st0);
            if constexpr (NW == 4) issue_w((uint32_t)qbase * gstride, w0);
            step(0, IntC<0>{}, std::false_type{});
            step(1, IntC<1>{}, std::false_type{});
            int v = 2;
#pragma clang loop unroll(disable)
            for (; v + L <= vend; v += L)
                static_for<0, L>([&](auto ic) __attribute__((always_inline)) {
                    constexpr int i = decltype(ic)::value;
                    step(v + i, IntC<2 + i>{}, std::true_type{});
                });
            auto tail = [&](auto self, auto ic) __attribute__((always_inline)) {
                constexpr int i = decltype(ic)::value;
                if constexpr (i + 1 < L) {
                    if (v + i < vend) {
                        step(v + i, IntC<2 + i>{}, std::true_type{});
                        self(self, IntC<i + 1>{});
                    }
                }
            };
            tail(tail, IntC<0>{});
            wait_vm<0>();   // the re-reads past the last block have landed
            // Every wave is done with the ring before the next pipeline refills it.
            stage_barrier();
            epilogue(qbase + qn - 1);
            };
            if constexpr (kChain) {
                pipeline(0, gn);
            } else {
                for (int q = 0; q < gn; ++q) pipeline(q, 1);
            }
        };
#if CAEE_P8_EVEN
        switch ((nb + 1) >> 1) {
            case 1: run(IntC<2>{}); break;
            case 2: run(IntC<4>{}); break;
            case 3: run(IntC<6>{}); break;
            case 4: run(IntC<8>{}); break;
            case 5: run(IntC<10>{}); break;
            case 6: run(IntC<12>{}); break;
            case 7: run(IntC<14>{}); break;
            default: run(IntC<16>{}); break;
        }
#else
        switch (nb) {
            case 1: run(IntC<1>{}); break;
            case 2: run(IntC<2>{}); break;
            case 3: run(IntC<3>{}); break;
            case 4: run(IntC<4>{}); break;
            case 5: run(IntC<5>{}); break;
            case 6: run(IntC<6>{}); break;
            case 7: run(IntC<7>{}); break;
            case 8: run(IntC<8>{}); break;
            case 9: run(IntC<9>{}); break;
            case 10: run(IntC<10>{}); break;
            case 11: run(IntC<11>{}); break;
            case 12: run(IntC<12>{}); break;
            case 13: run(IntC<13>{}); break;
            case 14: run(IntC<14>{}); break;
            case 15: run(IntC<15>{}); break;
            default: run(IntC<16>{}); break;
        }
#endif
    }
#endif
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

// The buffers the kernel reads through buffer descriptors (token codes and
// block scales of x and of the SwiGLU rows) must hold fewer than 2^31 bytes.
static bool p8_buffers_fit(long long T, long long P, long long d, long long f) {
    const long long lim = 1LL << 31;
    return T * d < lim && P * f < lim && (d / 128) * P * 4 < lim && (f / 128) * P * 4 < lim;
}

bool gemm_fp8_supports(const FfnParams& p, int nb) {
    return nb == kP8NT && p.tiled && p.f % 128 == 0 && p.d % 256 == 0 && p.d / 128 <= kP8MaxKBlocks &&
           p.f / 128 <= kP8MaxKBlocks && p8_buffers_fit(p.T, p.P, p.d, p.f);
}

bool gemm_fp8_applies(const caee_layer_desc_t& d, bool tiled) {
    return kGemmT > 0 && d.w_dtype == CAEE_FP8_E4M3 && d.T > kGemmT && tiled && d.f % 128 == 0 &&
           d.d % 256 == 0 && d.d / 128 <= kP8MaxKBlocks && d.f / 128 <= kP8MaxKBlocks &&
           p8_buffers_fit(d.T, (long long)d.T * (d.k + d.n_shared), d.d, d.f);
}

int gemm_fp8_blocks() { return kP8NT; }

bool gemm_fp8_fuses_quant() { return true; }

hipError_t launch_prefill8(const FfnParams& p, bool gate_up, int max_chunks, hipStream_t s) {
    const int groups = gate_up ? p.f / 128 : p.d / 256;
    // One workgroup per CU at a time (the ring takes most of the LDS); two
    // per CU in the grid, so that a CU whose items end early takes more.
    long long items = (long long)max_chunks * groups;
    const long long cap = (long long)device_cu_count() * CAEE_P8_GRID_PER_CU;
    if (items > cap) items = cap;
    if (items < 1) items = 1;
    if (gate_up) ffn_launch(k_prefill8<true>, dim3((unsigned)items), dim3(kP8Threads), s, p);
    else ffn_launch(k_prefill8<false>, dim3((unsigned)items), dim3(kP8Threads), s, p);
    return hipGetLastError();
}

}  // namespace caee
