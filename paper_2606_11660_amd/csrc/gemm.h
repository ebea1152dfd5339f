// Block-tile GEMM core for gfx950: C[m][n] += sum_k A[m][k] * B[n][k] with
// both operands K-contiguous rows (A: [M, K], B: [N, K]), fp16 or bf16
// inputs, fp32 accumulation on 16x16x32 MFMA.
//
// One workgroup (4 waves, 2 x 2) owns a 256 x 256 tile of C; each wave holds
// a 128 x 128 sub-tile as 8 x 8 MFMA accumulators (256 accumulator
// registers).  K advances in stages of 64 (128 bytes per row): every stage of
// A and B (32 KB each) is loaded with line-coalesced 16-byte loads (8 lanes
// per 128-byte row segment), parked in registers while the previous stage
// computes, and written to an XOR-swizzled LDS buffer (chunk ^ row % 8) from
// which MFMA fragments are read without bank conflicts.  Two LDS buffers,
// one barrier per stage.  Rows outside [0, M) / [0, N) read as zeros through
// the buffer resources' range check.
#pragma once

#include "common.h"

namespace attr {

constexpr int GT = 256;         // block tile (rows of A and of B)
constexpr int GK = 64;          // K per stage (elements; 128 bytes)
constexpr int G_STAGE_BYTES = GT * 128;  // one operand, one stage

struct GemmSmem {
  i32x4 a[2][GT * 8];
  i32x4 b[2][GT * 8];
};

template <typename Tag>
struct GemmCore {
  f32x4 acc[8][8];

  __device__ inline void zero() {
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  __device__ inline void scale(float s) {
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[i][j] *= s;
  }

  // Accumulate K in [0, n_stage * 64) of rows (a rows rsrc ra, stride lda
  // elements; b rows rsrc rb, stride ldb).  Both resources start at the
  // tile's first row.
  __device__ inline void run(GemmSmem& sm, __amdgpu_buffer_rsrc_t ra, int64_t lda,
                             __amdgpu_buffer_rsrc_t rb, int64_t ldb, int n_stage) {
    const int t = threadIdx.x;
    const int wave = t >> 6, lane = t & 63;
    const int wm = wave >> 1, wn = wave & 1;
    // load mapping: instruction j (0..7) of a wave covers rows 64 wave + 8 j + lane / 8
    const int lrow = lane >> 3, lch = lane & 7;
    const uint32_t a_off0 = (uint32_t)((int64_t)(64 * wave + lrow) * lda * 2 + lch * 16);
    const uint32_t b_off0 = (uint32_t)((int64_t)(64 * wave + lrow) * ldb * 2 + lch * 16);
    const uint32_t a_step8 = (uint32_t)(8 * lda * 2), b_step8 = (uint32_t)(8 * ldb * 2);
    // LDS slots written by this lane (row r = 64 wave + 8 j + lrow, r % 8 == lrow)
    const int wslot0 = (64 * wave + lrow) * 8 + (lch ^ lrow);
    // fragment read slots
    const int ri = lane & 15, rg = lane >> 4;

    i32x4 ga[8], gb[8];
    auto gload = [&](int st) {
      const uint32_t ko = (uint32_t)st * 128u;
#pragma unroll
      for (int j = 0; j < 8; ++j) ga[j] = load16_cached(ra, a_off0 + j * a_step8 + ko);
#pragma unroll
      for (int j = 0; j < 8; ++j) gb[j] = load16_cached(rb, b_off0 + j * b_step8 + ko);
    };
    auto lstore = [&](int buf) {
#pragma unroll
      for (int j = 0; j < 8; ++j) sm.a[buf][wslot0 + j * 64] = ga[j];
#pragma unroll
      for (int j = 0; j < 8; ++j) sm.b[buf][wslot0 + j * 64] = gb[j];
    };
    auto compute = [&](int buf) {
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        i32x4 fa[8], fb[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int row = 128 * wm + 16 * i + ri;
          fa[i] = sm.a[buf][row * 8 + ((4 * s + rg) ^ (row & 7))];
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int row = 128 * wn + 16 * j + ri;
          fb[j] = sm.b[buf][row * 8 + ((4 * s + rg) ^ (row & 7))];
        }
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
          for (int j = 0; j < 8; ++j) acc[i][j] = mma16(Tag{}, fa[i], fb[j], acc[i][j]);
      }
    };

    if (n_stage <= 0) return;
    gload(0);
    lstore(0);
    __syncthreads();
    for (int st = 0; st < n_stage; ++st) {
      const bool more = st + 1 < n_stage;
      if (more) gload(st + 1);
      compute(st & 1);
      if (more) lstore((st + 1) & 1);
      __syncthreads();
    }
  }

  // Row / column of accumulator element (i, j, r) for this lane.
  __device__ static inline int row_of(int i, int r) {
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    return 128 * (wave >> 1) + 16 * i + 4 * (lane >> 4) + r;
  }
  __device__ static inline int col_of(int j) {
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    return 128 * (wave & 1) + 16 * j + (lane & 15);
  }
};

}  // namespace attr
