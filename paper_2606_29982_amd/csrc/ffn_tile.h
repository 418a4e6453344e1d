// Tile contraction of the expert FFN kernels: the MFMA step of each weight
// format, the register-pipelined 16-row tile contraction and the SwiGLU
// row store.  Included inside namespace caee { namespace { ... } } by every
// translation unit that runs expert gate/up or down tiles.
#pragma once

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

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


__device__ inline float silu_mul(float g, float u) { return g / (1.0f + __expf(-g)) * u; }

// Loads through global-address-space pointers compile to global_load
// (a flat_load would also count against the LDS wait counter).
typedef const __attribute__((address_space(1))) u32x4_t g_u32x4_t;
__device__ inline u32x4_t load_stream(const u32x4_t* p) { return __builtin_nontemporal_load((g_u32x4_t*)p); }
__device__ inline u32x4_t load_cached(const u32x4_t* p) { return *(g_u32x4_t*)p; }

// Contraction of one 16-row weight tile against up to NB 16-token blocks,
// over `nsteps` k-steps starting at the given pointers, weights loaded U
// steps ahead of the MFMAs that consume them.  kTail: nsteps need not be a
// multiple of U; steps past the end are not multiplied.  Token blocks past
// nb read a valid row and are not multiplied.
//
// One token block (decode batches): both operands go into two register
// buffers used in turn, with no copies between them (a copy would have to
// wait for the loads it copies), and every batch of loads is issued
// unconditionally (steps at or past nsteps read the first activation piece:
// in bounds, in L2, never multiplied).  The wait before a batch of MFMAs is
// then for that batch's own loads only, and each wave keeps the next batch
// in flight while it multiplies.
//
// More token blocks: the activation pieces are loaded next to the MFMAs
// (double-buffering them too costs the kernel a resident wave per SIMD).
template <class M, int U, int NA, int NB, bool kTail, bool kAhead>
__device__ inline void tile_contract_steps(const u32x4_t* const (&a)[NA], int astep, const u32x4_t* const (&b)[NB],
                                           int nb, int nsteps, f32x4_t (&acc)[NA][NB]) {
    if constexpr (kAhead) {
        auto load = [&](u32x4_t (&w)[NA][U], u32x4_t (&x)[NB][U], int s) __attribute__((always_inline)) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int st = s + u;
                const bool in = st < nsteps;
#pragma unroll
                for (int m = 0; m < NA; ++m) w[m][u] = load_stream(in ? a[m] + (size_t)astep * st : b[0]);
#pragma unroll
                for (int tb = 0; tb < NB; ++tb) x[tb][u] = load_cached(in ? b[tb] + 4 * st : b[0]);
            }
        };
        auto mul = [&](const u32x4_t (&w)[NA][U], const u32x4_t (&x)[NB][U], int s) __attribute__((always_inline)) {
#pragma unroll
            for (int tb = 0; tb < NB; ++tb) {
                if (tb < nb) {
#pragma unroll
                    for (int u = 0; u < U; ++u) {
                        if (!kTail || s + u < nsteps) {
#pragma unroll
                            for (int m = 0; m < NA; ++m) M::mma(acc[m][tb], w[m][u], x[tb][u]);
                        }
                    }
                }
            }
        };
        u32x4_t w0[NA][U], x0[NB][U], w1[NA][U], x1[NB][U];
        load(w0, x0, 0);
        for (int ks = 0; ks < nsteps; ks += 2 * U) {
            load(w1, x1, ks + U);
            mul(w0, x0, ks);
            if (ks + U >= nsteps) break;
            load(w0, x0, ks + 2 * U);
            mul(w1, x1, ks + U);
        }
    } else {
        auto in_row = [&](int st) { return !kTail || st < nsteps ? st : nsteps - 1; };
        u32x4_t cur[NA][U], nxt[NA][U];
#pragma unroll
        for (int m = 0; m < NA; ++m)
#pragma unroll
            for (int u = 0; u < U; ++u) cur[m][u] = load_stream(a[m] + (size_t)astep * in_row(u));
        for (int ks = 0; ks < nsteps; ks += U) {
            const bool more = ks + U < nsteps;
            if (more) {
#pragma unroll
                for (int m = 0; m < NA; ++m)
#pragma unroll
                    for (int u = 0; u < U; ++u) nxt[m][u] = load_stream(a[m] + (size_t)astep * in_row(ks + U + u));
            }
#pragma unroll
            for (int tb = 0; tb < NB; ++tb) {
                if (tb < nb) {
#pragma unroll
                    for (int u = 0; u < U; ++u) {
                        if (!kTail || ks + u < nsteps) {
                            const u32x4_t bv = load_cached(b[tb] + 4 * (ks + u));
#pragma unroll
                            for (int m = 0; m < NA; ++m) M::mma(acc[m][tb], cur[m][u], bv);
                        }
                    }
                }
            }
            if (more) {
#pragma unroll
                for (int m = 0; m < NA; ++m)
#pragma unroll
                    for (int u = 0; u < U; ++u) cur[m][u] = nxt[m][u];
            }
        }
    }
}

template <class M, int U, int NA, int NB, bool kAhead = (NB == 1)>
__device__ inline void tile_contract(const u32x4_t* const (&a)[NA], int astep, const u32x4_t* const (&b)[NB],
                                     int nb, int nsteps, f32x4_t (&acc)[NA][NB]) {
    if (nsteps % U == 0) tile_contract_steps<M, U, NA, NB, false, kAhead>(a, astep, b, nb, nsteps, acc);
    else tile_contract_steps<M, U, NA, NB, true, kAhead>(a, astep, b, nb, nsteps, acc);
}

template <class M>
__device__ inline void store_h(const FfnParams& p, size_t o, const float (&h)[4]) {
    if (M::kElemBytes == 2) {
        uint2 pk;
        pk.x = bf16_rne(h[0]) | (bf16_rne(h[1]) << 16);
        pk.y = bf16_rne(h[2]) | (bf16_rne(h[3]) << 16);
        *(uint2*)((uint16_t*)p.h + o) = pk;
    } else {
        *(float4*)((float*)p.h + o) = make_float4(h[0], h[1], h[2], h[3]);
    }
}
