// Staging of activation rows into LDS for the big-chunk FFN kernels
// (shared by the 16-bit and 8-bit paths).
//
// A stage is 256 bytes of each of a chunk's up to 16*NB token rows: four
// 64-byte contraction steps of the 16-bit MFMA, or two 128-wide blocks of the
// 8-bit one.  Thread `tid` of the 256-thread workgroup moves the 16-byte
// piece q = tid % 16 of token tid / 16 + 16 j for every token block j.  In
// LDS a stage is [token block][step][lane] 16-byte pieces, lane l = r + 16 g
// holding bytes [16 g, 16 g + 16) of step `step` of token 16 j + r: exactly
// the B fragment lane l of an MFMA reads, so each fragment is one
// conflict-free 16-byte LDS load.
#pragma once

#include "caee_internal.h"

namespace caee {

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kStageSteps = 4;   // 64-byte steps per stage
constexpr int kStagePieces = 16; // 16-byte pieces per token row per stage

template <int NB>
struct RowStage {
    const u32x4_t* src[NB];      // this thread's piece of each token row's first stage
    int q;                       // piece index within the stage
    __device__ inline void init(const u32x4_t* const (&rows)[NB], int tid) {
        q = tid & (kStagePieces - 1);
#pragma unroll
        for (int j = 0; j < NB; ++j) src[j] = rows[j] + q;
    }
    // Pieces at or past `row_pieces` (the row's length) are not read.
    __device__ inline void load(u32x4_t (&v)[NB], int kb, int nb, int row_pieces) const {
        const bool in = kb * kStagePieces + q < row_pieces;
#pragma unroll
        for (int j = 0; j < NB; ++j)
            if (j < nb && in) v[j] = src[j][(size_t)kb * kStagePieces];
    }
    __device__ inline void store(u32x4_t (*sb)[kStageSteps][kWave], const u32x4_t (&v)[NB], int tid, int nb,
                                 int kb, int row_pieces) const {
        const int l = (tid >> 4) + 16 * (q & 3), step = q >> 2;
        const bool in = kb * kStagePieces + q < row_pieces;
#pragma unroll
        for (int j = 0; j < NB; ++j)
            if (j < nb && in) sb[j][step][l] = v[j];
    }
};

}  // namespace caee
