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

namespace caee {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kNB = kChunkTokens / 16;   // 16-token MFMA column blocks per chunk

// One 16-byte load per lane = one contraction step of the 16x16 MFMA tile.
struct Bf16Math {
    static constexpr int kElemBytes = 2;
    __device__ static inline void mma(f32x4_t& acc, const u32x4_t& a, const u32x4_t& b) {
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                      __builtin_bit_cast(bf16x8_t, b), acc, 0, 0, 0);
    }
};

struct F32Math {
    static constexpr int kElemBytes = 4;
    __device__ static inline void mma(f32x4_t& acc, const u32x4_t& a, const u32x4_t& b) {
#pragma unroll
        for (int u = 0; u < 4; ++u)
            acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[u]), __uint_as_float(b[u]), acc,
                                                       0, 0, 0);
    }
};

__device__ inline uint32_t bf16_rne(float v) {
    const uint32_t u = __float_as_uint(v);
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

__device__ inline float silu_mul(float g, float u) { return g / (1.0f + __expf(-g)) * u; }

__device__ inline const char* expert_base(const void* routed, const void* shared, int x, int E,
                                          size_t expert_bytes) {
    return x < E ? (const char*)routed + (size_t)x * expert_bytes
                 : (const char*)shared + (size_t)(x - E) * expert_bytes;
}

template <class M, int U>
__global__ __launch_bounds__(kFfnThreads) void k_gate_up(FfnParams p) {
    const int lane = threadIdx.x & (kWave - 1);
    const int r = lane & 15, g = lane >> 4;
    const int gw = blockIdx.x * (kFfnThreads / kWave) + (threadIdx.x / kWave);
    const int nw = gridDim.x * (kFfnThreads / kWave);
    const int tiles = p.f / 16;
    const int total = (*p.n_chunks) * tiles;
    const size_t row_units = (size_t)p.d * M::kElemBytes / 16;
    const int ksteps = (int)(row_units / 4);
    const size_t expert_bytes = (size_t)2 * p.f * p.d * M::kElemBytes;

    for (int item = gw; item < total; item += nw) {
        const int c = item / tiles, jt = item - c * tiles;
        const int xs = p.chunks[4 * c], row0 = p.chunks[4 * c + 1], ntok = p.chunks[4 * c + 2];
        const u32x4_t* wb = (const u32x4_t*)expert_base(p.w13, p.sh_w13, xs, p.E, expert_bytes);
        const u32x4_t* ag = wb + (size_t)(jt * 16 + r) * row_units + g;
        const u32x4_t* au = wb + (size_t)(p.f + jt * 16 + r) * row_units + g;
        const int nb = (ntok + 15) >> 4;
        const u32x4_t* xb[kNB];
#pragma unroll
        for (int tb = 0; tb < kNB; ++tb) {
            int n = tb * 16 + r;
            n = n < ntok ? n : 0;   // padded token columns read a valid row; their results are dropped
            xb[tb] = (const u32x4_t*)p.x + (size_t)p.perm_tok[row0 + n] * row_units + g;
        }
        f32x4_t accg[kNB], accu[kNB];
#pragma unroll
        for (int tb = 0; tb < kNB; ++tb) {
            accg[tb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
            accu[tb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        }
        for (int ks = 0; ks < ksteps; ks += U) {
            u32x4_t a0[U], a1[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                a0[u] = __builtin_nontemporal_load(ag + 4 * (ks + u));
                a1[u] = __builtin_nontemporal_load(au + 4 * (ks + u));
            }
#pragma unroll
            for (int tb = 0; tb < kNB; ++tb) {
                if (tb < nb) {
#pragma unroll
                    for (int u = 0; u < U; ++u) {
                        const u32x4_t b = xb[tb][4 * (ks + u)];
                        M::mma(accg[tb], a0[u], b);
                        M::mma(accu[tb], a1[u], b);
                    }
                }
            }
        }
        // Lane holds rows 4g..4g+3 of the tile (intermediate features) for token column r.
#pragma unroll
        for (int tb = 0; tb < kNB; ++tb) {
            const int n = tb * 16 + r;
            if (tb < nb && n < ntok) {
                const size_t o = (size_t)(row0 + n) * p.f + jt * 16 + 4 * g;
                float h[4];
#pragma unroll
                for (int v = 0; v < 4; ++v) h[v] = silu_mul(accg[tb][v], accu[tb][v]);
                if (M::kElemBytes == 2) {
                    uint2 pk;
                    pk.x = bf16_rne(h[0]) | (bf16_rne(h[1]) << 16);
                    pk.y = bf16_rne(h[2]) | (bf16_rne(h[3]) << 16);
                    *(uint2*)((uint16_t*)p.h + o) = pk;
                } else {
                    *(float4*)((float*)p.h + o) = make_float4(h[0], h[1], h[2], h[3]);
                }
            }
        }
    }
}

template <class M, int U>
__global__ __launch_bounds__(kFfnThreads) void k_down(FfnParams p) {
    const int lane = threadIdx.x & (kWave - 1);
    const int r = lane & 15, g = lane >> 4;
    const int gw = blockIdx.x * (kFfnThreads / kWave) + (threadIdx.x / kWave);
    const int nw = gridDim.x * (kFfnThreads / kWave);
    const int tiles = p.d / 16;
    const int total = (*p.n_chunks) * tiles;
    const size_t row_units = (size_t)p.f * M::kElemBytes / 16;
    const int ksteps = (int)(row_units / 4);
    const size_t expert_bytes = (size_t)p.d * p.f * M::kElemBytes;

    for (int item = gw; item < total; item += nw) {
        const int c = item / tiles, it = item - c * tiles;
        const int xs = p.chunks[4 * c], row0 = p.chunks[4 * c + 1], ntok = p.chunks[4 * c + 2];
        const u32x4_t* wb = (const u32x4_t*)expert_base(p.w2, p.sh_w2, xs, p.E, expert_bytes);
        const u32x4_t* a = wb + (size_t)(it * 16 + r) * row_units + g;
        const int nb = (ntok + 15) >> 4;
        const u32x4_t* hb[kNB];
#pragma unroll
        for (int tb = 0; tb < kNB; ++tb) {
            int n = tb * 16 + r;
            n = n < ntok ? n : 0;
            hb[tb] = (const u32x4_t*)p.h + (size_t)(row0 + n) * row_units + g;
        }
        f32x4_t acc[kNB];
#pragma unroll
        for (int tb = 0; tb < kNB; ++tb) acc[tb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        for (int ks = 0; ks < ksteps; ks += U) {
            u32x4_t aw[U];
#pragma unroll
            for (int u = 0; u < U; ++u) aw[u] = __builtin_nontemporal_load(a + 4 * (ks + u));
#pragma unroll
            for (int tb = 0; tb < kNB; ++tb) {
                if (tb < nb) {
#pragma unroll
                    for (int u = 0; u < U; ++u) M::mma(acc[tb], aw[u], hb[tb][4 * (ks + u)]);
                }
            }
        }
#pragma unroll
        for (int tb = 0; tb < kNB; ++tb) {
            const int n = tb * 16 + r;
            if (tb < nb && n < ntok) {
                float* o = p.yperm + (size_t)(row0 + n) * p.d + it * 16 + 4 * g;
                *(float4*)o = make_float4(acc[tb][0], acc[tb][1], acc[tb][2], acc[tb][3]);
            }
        }
    }
}

// One thread per 4 output features of one token.
__global__ __launch_bounds__(256) void k_combine(FfnParams p) {
    const int t = blockIdx.y;
    const int c = (blockIdx.x * 256 + threadIdx.x) * 4;
    if (c >= p.d) return;
    const int slots = p.k + p.n_shared;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int j = 0; j < p.k; ++j) {
        const int pos = p.perm_pos[t * slots + j];
        if (pos < 0) continue;
        const float w = p.topk_w[t * p.k + j];
        const float4 v = *(const float4*)(p.yperm + (size_t)pos * p.d + c);
        acc.x = fmaf(w, v.x, acc.x);
        acc.y = fmaf(w, v.y, acc.y);
        acc.z = fmaf(w, v.z, acc.z);
        acc.w = fmaf(w, v.w, acc.w);
    }
    for (int s = 0; s < p.n_shared; ++s) {
        const int pos = p.perm_pos[t * slots + p.k + s];
        const float4 v = *(const float4*)(p.yperm + (size_t)pos * p.d + c);
        acc.x += v.x;
        acc.y += v.y;
        acc.z += v.z;
        acc.w += v.w;
    }
    const size_t o = (size_t)t * p.d + c;
    if (p.y_bf16) {
        uint2 pk;
        pk.x = bf16_rne(acc.x) | (bf16_rne(acc.y) << 16);
        pk.y = bf16_rne(acc.z) | (bf16_rne(acc.w) << 16);
        *(uint2*)((uint16_t*)p.y + o) = pk;
    } else {
        *(float4*)((float*)p.y + o) = acc;
    }
}

int grid_for(long long waves_needed) {
    const long long wgs = (waves_needed + 3) / 4;
    const long long cap = (long long)device_cu_count() * 8;
    return (int)(wgs < 1 ? 1 : (wgs < cap ? wgs : cap));
}

}  // namespace

hipError_t launch_gate_up(const FfnParams& p, int w_dtype, int max_chunks, hipStream_t s) {
    const dim3 grid(grid_for((long long)max_chunks * (p.f / 16)));
    if (w_dtype == CAEE_BF16)
        hipLaunchKernelGGL((k_gate_up<Bf16Math, 4>), grid, dim3(kFfnThreads), 0, s, p);
    else if (w_dtype == CAEE_F32)
        hipLaunchKernelGGL((k_gate_up<F32Math, 4>), grid, dim3(kFfnThreads), 0, s, p);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

hipError_t launch_down(const FfnParams& p, int w_dtype, int max_chunks, hipStream_t s) {
    const dim3 grid(grid_for((long long)max_chunks * (p.d / 16)));
    if (w_dtype == CAEE_BF16)
        hipLaunchKernelGGL((k_down<Bf16Math, 4>), grid, dim3(kFfnThreads), 0, s, p);
    else if (w_dtype == CAEE_F32)
        hipLaunchKernelGGL((k_down<F32Math, 4>), grid, dim3(kFfnThreads), 0, s, p);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

hipError_t launch_combine(const FfnParams& p, hipStream_t s) {
    const dim3 grid((p.d / 4 + 255) / 256, p.T);
    hipLaunchKernelGGL(k_combine, grid, dim3(256), 0, s, p);
    return hipGetLastError();
}

}  // namespace caee
