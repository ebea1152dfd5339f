// Block-tile GEMM core for gfx950: C[m][n] += sum_k A[m][k] * B[n][k] with
// both operands K-contiguous rows (A: [M, K], B: [N, K]), fp16 or bf16
// inputs, fp32 accumulation on 16x16x32 MFMA.
//
// One workgroup (4 waves, 2 x 2) owns a 256 x 256 tile of C; each wave holds
// a 128 x 128 sub-tile as 8 x 8 MFMA accumulators (256 accumulator
// registers).  K advances in stages of 64 (128 bytes per row).  Every stage of
// A and B (32 KB each) goes from memory straight into one of two LDS slots by
// direct-to-LDS buffer loads (8 rows x 128 bytes per instruction, 16
// instructions per wave and stage), so no operand passes through registers
// on its way to LDS and no wave spends instructions on LDS stores.  In LDS a
// row is 128 bytes; its 16-byte chunk c sits in slot c ^ (row % 8), which the
// loads produce by fetching the permuted chunk, so that the MFMA fragment
// reads hit distinct bank groups.
//
// A stage is consumed as two K-halves, h0 and h1, each 64 MFMAs from 16
// fragments held in registers (two fragment sets).  The step of stage s
// runs: wait for stage s, barrier (stage s visible to every
// wave; every wave has finished reading stage s - 1, whose slot is then
// refilled with stage s + 1), then the MFMAs of h1 of stage s - 1 while the
// fragments of h0 of stage s are read, then the MFMAs of h0 of stage s while
// the fragments of h1 of stage s are read.  The 16 loads of stage s + 1 are
// spread over the first 64 MFMAs of the step (one per 4: late enough not to
// fill the address queue in one burst, early enough to land before the next
// step), the 32 fragment reads over all 128 (two per 8): issued in bursts
// they fill the address and LDS command queues and stall the wave, and with
// it the matrix core.  Rows outside the operand's
// range read as zeros through the buffer descriptors' range check.  NT loads
// B with the non-temporal cache policy, for a B that is read once (a stream
// of store rows against a single tile of queries).
#pragma once

#include <type_traits>

#include "common.h"

namespace attr {

constexpr int GT = 256;                  // block tile (rows of A and of B)
constexpr int GKS = 64;                  // K per stage (elements; 128 bytes)
constexpr uint32_t G_SLOT = GT * 128;    // bytes per operand per slot

struct GemmSmem {
  i32x4 a[2][GT * 8];
  i32x4 b[2][GT * 8];
};

template <int N>
__device__ inline void gemm_wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

template <typename Tag, bool NT = false>
struct GemmCore {
  f32x4 acc[8][8];

  __device__ inline void zero() {
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // Accumulate n_st stages (K = 64 n_st) of the tile's rows: A rows through
  // descriptor da (row stride lda elements), B rows through db (stride ldb);
  // both descriptors start at the tile's first row.  Byte offsets within a
  // descriptor must fit 31 bits.
  __device__ inline void run(GemmSmem& sm, const i32x4& da, int64_t lda, const i32x4& db,
                             int64_t ldb, int n_st) {
    if (n_st <= 0) return;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int lane = threadIdx.x & 63;
    const int wm = wave >> 1, wn = wave & 1;
    // loads: instruction h (0..7) of a wave covers rows 64 wave + 8 h + lane / 8;
    // the lane's LDS slot (lane % 8) receives chunk (lane % 8) ^ (lane / 8)
    const int lr = lane >> 3;
    const int lc = (lane & 7) ^ lr;
    const uint32_t a_off = (uint32_t)((int64_t)(64 * wave + lr) * lda * 2 + lc * 16);
    const uint32_t b_off = (uint32_t)((int64_t)(64 * wave + lr) * ldb * 2 + lc * 16);
    const uint32_t a8 = (uint32_t)(8 * lda * 2), b8 = (uint32_t)(8 * ldb * 2);
    const uint32_t lds_a = (uint32_t)(uintptr_t)&sm.a[0][0] + (uint32_t)(64 * wave) * 128u;
    const uint32_t lds_b = (uint32_t)(uintptr_t)&sm.b[0][0] + (uint32_t)(64 * wave) * 128u;
    // loads of stage st come in 4 groups of 4 instructions (A rows 0-31 and
    // 32-63 of the wave, then B): group g sets M0 once, instruction u of it
    // lands at M0 + 1024 u through the instruction offset.  The stage's K
    // offset moves the descriptors (desc_at), so the per-lane offsets are
    // fixed.  A stage past the end is issued with every lane out of range:
    // it fetches nothing and zero-fills a slot that is no longer read.
    auto issue_grp = [&](int slot, int g) {
      set_m0((g < 2 ? lds_a : lds_b) + (uint32_t)slot * G_SLOT + (uint32_t)(g & 1) * 4096u);
    };
    auto issue_u = [&](int st, int g, auto uc) {
      constexpr int u = decltype(uc)::value;
      const int h = 4 * (g & 1) + u;
      const uint32_t ko = (uint32_t)st * 128u;
      const bool live = st < n_st;
      if (g < 2) {
        lds_dma16_m0<1024 * u>(desc_at(da, ko, live), a_off + h * a8 - 1024u * u);
      } else if (NT) {
        lds_dma16_m0_nt<1024 * u>(desc_at(db, ko, live), b_off + h * b8 - 1024u * u);
      } else {
        lds_dma16_m0<1024 * u>(desc_at(db, ko, live), b_off + h * b8 - 1024u * u);
      }
    };
    auto issue_all = [&](int st) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        issue_grp(st & 1, g);
        issue_u(st, g, std::integral_constant<int, 0>{});
        issue_u(st, g, std::integral_constant<int, 1>{});
        issue_u(st, g, std::integral_constant<int, 2>{});
        issue_u(st, g, std::integral_constant<int, 3>{});
      }
    };
    // fragment reads: lane (ri, rg) takes row 16 t + ri, chunk 4 half + rg in
    // slot (4 half + rg) ^ (ri % 8)
    const int ri = lane & 15, rg = lane >> 4;
    const int fa0 = (128 * wm + ri) * 8, fb0 = (128 * wn + ri) * 8;
    const int fs0 = rg ^ (ri & 7), fs1 = (4 + rg) ^ (ri & 7);
    // the 16 fragments of a half, two per call, B first: every MFMA row needs
    // all of B but only its own row of A
    auto read_pair = [&](int i, const i32x4* pa, const i32x4* pb, int fs, i32x4 (&fa)[8],
                         i32x4 (&fb)[8]) {
      if (i < 4) {
        fb[2 * i] = pb[fb0 + 128 * (2 * i) + fs];
        fb[2 * i + 1] = pb[fb0 + 128 * (2 * i + 1) + fs];
      } else {
        fa[2 * i - 8] = pa[fa0 + 128 * (2 * i - 8) + fs];
        fa[2 * i - 7] = pa[fa0 + 128 * (2 * i - 7) + fs];
      }
    };
    auto mma_row = [&](int i, const i32x4 (&fa)[8], const i32x4 (&fb)[8]) {
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[i][j] = mma16(Tag{}, fa[i], fb[j], acc[i][j]);
    };
    i32x4 h0a[8], h0b[8], h1a[8], h1b[8];

    // prologue: stage 0 in, stage 1 on its way, h0 of stage 0 in registers
    issue_all(0);
    gemm_wait_vm<0>();
    __builtin_amdgcn_s_barrier();
    issue_all(1);
    {
      const i32x4* pa = sm.a[0];
      const i32x4* pb = sm.b[0];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        h0a[i] = pa[fa0 + 128 * i + fs0];
        h0b[i] = pb[fb0 + 128 * i + fs0];
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        read_pair(i, pa, pb, fs1, h1a, h1b);
        __builtin_amdgcn_sched_barrier(0);
        mma_row(i, h0a, h0b);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    // stage st in slot SLOT = st & 1, a compile-time constant (the loop runs
    // in pairs), so the fragment reads carry the slot in their offset field
    auto stage = [&](int st, auto slot_c) {
      constexpr int SLOT = decltype(slot_c)::value;
      // stage st landed (nothing later is in flight); this wave's reads of
      // stage st - 1 are complete
      gemm_wait_vm<0>();
      wait_lgkm0();
      __builtin_amdgcn_s_barrier();
      const i32x4* pa = sm.a[SLOT];
      const i32x4* pb = sm.b[SLOT];
      // h1 of stage st - 1, reading h0 of stage st, loading stage st + 1
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        read_pair(i, pa, pb, fs0, h0a, h0b);
        // loads 2 i and 2 i + 1 of stage st + 1: group i / 2, members
        // 2 (i % 2) and 2 (i % 2) + 1
        if ((i & 1) == 0) {
          issue_grp(1 - SLOT, i >> 1);
          issue_u(st + 1, i >> 1, std::integral_constant<int, 0>{});
        } else {
          issue_u(st + 1, i >> 1, std::integral_constant<int, 2>{});
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = mma16(Tag{}, h1a[i], h1b[j], acc[i][j]);
        __builtin_amdgcn_sched_barrier(0);
        if ((i & 1) == 0) {
          issue_u(st + 1, i >> 1, std::integral_constant<int, 1>{});
        } else {
          issue_u(st + 1, i >> 1, std::integral_constant<int, 3>{});
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int j = 4; j < 8; ++j) acc[i][j] = mma16(Tag{}, h1a[i], h1b[j], acc[i][j]);
        __builtin_amdgcn_sched_barrier(0);
      }
      // h0 of stage st, reading h1 of stage st
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        read_pair(i, pa, pb, fs1, h1a, h1b);
        __builtin_amdgcn_sched_barrier(0);
        mma_row(i, h0a, h0b);
        __builtin_amdgcn_sched_barrier(0);
      }
    };
    int st = 1;
    for (; st + 1 < n_st; st += 2) {
      stage(st, std::integral_constant<int, 1>{});
      stage(st + 1, std::integral_constant<int, 0>{});
    }
    if (st < n_st) stage(st, std::integral_constant<int, 1>{});
    // h1 of the last stage
#pragma unroll
    for (int i = 0; i < 8; ++i) mma_row(i, h1a, h1b);
    // the zero-filling loads past the end have landed and every wave's LDS
    // reads are complete before the caller reuses the slots
    gemm_wait_vm<0>();
    wait_lgkm0();
    __builtin_amdgcn_s_barrier();
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
  static constexpr int NJ = 8;  // 16-column accumulator blocks per wave
  __device__ static inline int col_base() { return 128 * (int)((threadIdx.x >> 6) & 1); }
};

// The 256 x 256 tile of GemmCore for C = A (B1 + B2)^T with the two B
// operands interleaved per K-block: step 2 s multiplies A block s by B1
// block s, step 2 s + 1 the same A block by B2 block s (one accumulator).
// A block s is loaded into LDS once for both steps, with two steps to land
// (it is issued in step 2 s - 2, after that step's B load, into the A slot
// the pair before freed), and the odd step reuses the even step's A
// fragments from registers, so per pair of steps the core issues 24 loads
// and 48 fragment reads per wave instead of 32 and 64, and reads A from
// memory once instead of once per B operand.  Otherwise the pipeline is
// GemmCore's: wait for step t, barrier, MFMAs of h1 of step t - 1 while
// reading h0 of t, then MFMAs of h0 of t while reading h1 of t.
template <typename Tag>
struct GemmCoreHL {
  f32x4 acc[8][8];

  __device__ inline void zero() {
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // n_k K-blocks of 64 (2 n_k steps): A rows through da (stride lda), B1 and
  // B2 rows through db1, db2 (stride ldb), all from the tile's first row.
  // Rows outside a descriptor's range read as zeros; byte offsets must fit
  // 31 bits.
  __device__ inline void run(GemmSmem& sm, const i32x4& da, int64_t lda, const i32x4& db1,
                             const i32x4& db2, int64_t ldb, int n_k) {
    if (n_k <= 0) return;
    const int n_t = 2 * n_k;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int lane = threadIdx.x & 63;
    const int wm = wave >> 1, wn = wave & 1;
    const int lr = lane >> 3;
    const int lc = (lane & 7) ^ lr;
    const uint32_t a_off = (uint32_t)((int64_t)(64 * wave + lr) * lda * 2 + lc * 16);
    const uint32_t b_off = (uint32_t)((int64_t)(64 * wave + lr) * ldb * 2 + lc * 16);
    const uint32_t a8 = (uint32_t)(8 * lda * 2), b8 = (uint32_t)(8 * ldb * 2);
    const uint32_t lds_a = (uint32_t)(uintptr_t)&sm.a[0][0] + (uint32_t)(64 * wave) * 128u;
    const uint32_t lds_b = (uint32_t)(uintptr_t)&sm.b[0][0] + (uint32_t)(64 * wave) * 128u;
    // load n (0..7) of A block s (slot s & 1) or of B step t (slot t & 1):
    // group n / 4 covers rows 32 (n / 4) .. + 31 of the wave's 64, member
    // n % 4 lands at M0 + 1024 (n % 4); past the end nothing is fetched.
    auto load_a = [&](int s, int n) {
      const int g = n >> 2, u = n & 3;
      const i32x4 d = desc_at(da, (uint32_t)s * 128u, s < n_k);
      if (u == 0) set_m0(lds_a + (uint32_t)(s & 1) * G_SLOT + (uint32_t)g * 4096u);
      const uint32_t voff = a_off + (uint32_t)(4 * g + u) * a8;
      switch (u) {
        case 0: lds_dma16_m0<0>(d, voff); break;
        case 1: lds_dma16_m0<1024>(d, voff - 1024u); break;
        case 2: lds_dma16_m0<2048>(d, voff - 2048u); break;
        default: lds_dma16_m0<3072>(d, voff - 3072u); break;
      }
    };
    // d: db1 for even t, db2 for odd t (the caller knows the parity at
    // compile time: a run-time choice put a VALU write of the descriptor
    // right before the load)
    auto load_b = [&](int t, int n, const i32x4& db) {
      const int g = n >> 2, u = n & 3;
      const i32x4 d = desc_at(db, (uint32_t)(t >> 1) * 128u, t < n_t);
      if (u == 0) set_m0(lds_b + (uint32_t)(t & 1) * G_SLOT + (uint32_t)g * 4096u);
      const uint32_t voff = b_off + (uint32_t)(4 * g + u) * b8;
      switch (u) {
        case 0: lds_dma16_m0<0>(d, voff); break;
        case 1: lds_dma16_m0<1024>(d, voff - 1024u); break;
        case 2: lds_dma16_m0<2048>(d, voff - 2048u); break;
        default: lds_dma16_m0<3072>(d, voff - 3072u); break;
      }
    };
    const int ri = lane & 15, rg = lane >> 4;
    const int fa0 = (128 * wm + ri) * 8, fb0 = (128 * wn + ri) * 8;
    const int fs0 = rg ^ (ri & 7), fs1 = (4 + rg) ^ (ri & 7);
    // the fragments of a half, two per call (B first); RA: also A's
    auto read_pair = [&](int i, bool ra, const i32x4* pa, const i32x4* pb, int fs, i32x4 (&fa)[8],
                         i32x4 (&fb)[8]) {
      if (i < 4) {
        fb[2 * i] = pb[fb0 + 128 * (2 * i) + fs];
        fb[2 * i + 1] = pb[fb0 + 128 * (2 * i + 1) + fs];
      } else if (ra) {
        fa[2 * i - 8] = pa[fa0 + 128 * (2 * i - 8) + fs];
        fa[2 * i - 7] = pa[fa0 + 128 * (2 * i - 7) + fs];
      }
    };
    auto mma_row = [&](int i, const i32x4 (&fa)[8], const i32x4 (&fb)[8]) {
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[i][j] = mma16(Tag{}, fa[i], fb[j], acc[i][j]);
    };
    i32x4 h0a[8], h0b[8], h1a[8], h1b[8];

    // prologue: A block 0 and B step 0 in; B step 1 and A block 1 on their
    // way; h0 of step 0 in registers, then h1 of step 0 read under the MFMAs
    // of its h0
#pragma unroll
    for (int n = 0; n < 8; ++n) load_a(0, n);
#pragma unroll
    for (int n = 0; n < 8; ++n) load_b(0, n, db1);
    gemm_wait_vm<0>();
    __builtin_amdgcn_s_barrier();
#pragma unroll
    for (int n = 0; n < 8; ++n) load_b(1, n, db2);
#pragma unroll
    for (int n = 0; n < 8; ++n) load_a(1, n);
    {
      const i32x4* pa = sm.a[0];
      const i32x4* pb = sm.b[0];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        h0a[i] = pa[fa0 + 128 * i + fs0];
        h0b[i] = pb[fb0 + 128 * i + fs0];
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        read_pair(i, true, pa, pb, fs1, h1a, h1b);
        __builtin_amdgcn_sched_barrier(0);
        mma_row(i, h0a, h0b);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    // step t (t >= 1): ODD steps reuse the A fragments of step t - 1 and load
    // only B; even steps (t = 2 s) also load A block s + 1
    auto step = [&](int t, auto odd_c) {
      constexpr bool ODD = decltype(odd_c)::value;
      // odd: B of step t was issued before the A block that may still be in
      // flight (8 loads); even: everything issued before step t - 1's B
      if (ODD) {
        gemm_wait_vm<8>();
      } else {
        gemm_wait_vm<0>();
      }
      wait_lgkm0();
      __builtin_amdgcn_s_barrier();
      const i32x4* pa = sm.a[(t >> 1) & 1];
      const i32x4* pb = sm.b[t & 1];
      // h1 of step t - 1, reading h0 of step t, loading B of step t + 1 (odd:
      // one load per row; even: all of B in rows 0-3, then A block t / 2 + 1
      // in rows 4-7, so that every B load precedes every A load and the odd
      // step's wait leaves exactly the 8 A loads in flight)
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        read_pair(i, !ODD, pa, pb, fs0, h0a, h0b);
        if (ODD) {
          load_b(t + 1, i, db1);
        } else if (i < 4) {
          load_b(t + 1, 2 * i, db2);
        } else {
          load_a((t >> 1) + 1, 2 * (i - 4));
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = mma16(Tag{}, h1a[i], h1b[j], acc[i][j]);
        __builtin_amdgcn_sched_barrier(0);
        if (!ODD) {
          if (i < 4) {
            load_b(t + 1, 2 * i + 1, db2);
          } else {
            load_a((t >> 1) + 1, 2 * (i - 4) + 1);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int j = 4; j < 8; ++j) acc[i][j] = mma16(Tag{}, h1a[i], h1b[j], acc[i][j]);
        __builtin_amdgcn_sched_barrier(0);
      }
      // h0 of step t, reading h1 of step t
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        read_pair(i, !ODD, pa, pb, fs1, h1a, h1b);
        __builtin_amdgcn_sched_barrier(0);
        mma_row(i, h0a, h0b);
        __builtin_amdgcn_sched_barrier(0);
      }
    };
    for (int t = 1; t < n_t; t += 2) {
      step(t, std::integral_constant<bool, true>{});
      if (t + 1 < n_t) step(t + 1, std::integral_constant<bool, false>{});
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) mma_row(i, h1a, h1b);
    gemm_wait_vm<0>();
    wait_lgkm0();
    __builtin_amdgcn_s_barrier();
  }
};

// Query-narrow ring tile: 128 rows of A (queries) against 256 rows of B
// (store rows) with a three-slot LDS ring, for streaming a large B past a
// small A.  Wave w holds all 128 A rows against B rows [64 w, 64 w + 64) as
// 8 x 4 MFMA accumulators.  A slot holds one stage (K = 64): 16 KB of A and
// 32 KB of B (144 KB for the ring).  The step of stage s waits only for
// stage s (the loads of stage s + 1 stay in flight), crosses the barrier
// (stage s visible; the slot of stage s - 1 free) and refills that slot with
// stage s + 2 while the MFMAs run, so two stages are always on their way
// from memory and the issue never drains: at one workgroup per CU a ring of
// 256-row x 128-byte stages streams at ~7.1 TB/s, where waiting for every
// load before issuing the next stage (the two-slot schedule) holds a read
// stream to ~5 TB/s.  Each wave loads 4 KB of A and its own 8 KB of B per
// stage (12 direct-to-LDS loads, M0 set once per 4), one load per issue
// point over the first 12 of the 16 points of a step, and reads B through
// its own descriptor.  Fragment reads, the two K-halves and their register
// sets are GemmCore's.  NT loads B with the non-temporal cache policy (B
// read once): at 2M x 8192 store rows and 128 queries that took the whole
// scan from 6.42 to 5.64 ms (the data stream no longer competes with the
// queries, which every workgroup re-reads, for cache).
constexpr int GRQ = 128;                 // A rows per tile
constexpr int GRR = 256;                 // B rows per tile (64 per wave)
constexpr int GR_SLOTS = 3;

struct GemmSmemR {
  i32x4 a[GR_SLOTS][GRQ * 8];
  i32x4 b[GR_SLOTS][GRR * 8];
};

template <typename Tag, bool NT = false>
struct GemmCoreR {
  f32x4 acc[8][4];

  __device__ inline void zero() {
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // n_st stages (K = 64 n_st): da covers the tile's A rows (stride lda), dbw
  // this wave's 64 B rows (stride ldb), both from their first row.  Rows
  // outside a descriptor's range read as zeros; byte offsets fit 31 bits
  // when 128 rows of either operand span less than 1 GiB.
  __device__ inline void run(GemmSmemR& sm, const i32x4& da, int64_t lda, const i32x4& dbw,
                             int64_t ldb, int n_st) {
    if (n_st <= 0) return;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int lane = threadIdx.x & 63;
    const int lr = lane >> 3;
    const int lc = (lane & 7) ^ lr;
    // A: rows 32 wave + 8 u + lane / 8 (u = 0..3); B: the wave's rows
    // 8 (4 g + u) + lane / 8 (g = 0, 1; u = 0..3)
    const uint32_t a_off = (uint32_t)((int64_t)(32 * wave + lr) * lda * 2 + lc * 16);
    const uint32_t b_off = (uint32_t)((int64_t)lr * ldb * 2 + lc * 16);
    const uint32_t a8 = (uint32_t)(8 * lda * 2), b8 = (uint32_t)(8 * ldb * 2);
    const uint32_t lds_a = (uint32_t)(uintptr_t)&sm.a[0][0] + (uint32_t)(32 * wave) * 128u;
    const uint32_t lds_b = (uint32_t)(uintptr_t)&sm.b[0][0] + (uint32_t)(64 * wave) * 128u;
    constexpr uint32_t SLOT_A = GRQ * 128, SLOT_B = GRR * 128;
    // load n (0..11) of stage st into slot sl: group n / 4 (0: A, 1-2: B),
    // member n % 4; a stage past the end fetches nothing and zero-fills a
    // slot that is not read again
    auto issue = [&](int st, int sl, int n) {
      const int g = n >> 2, u = n & 3;
      const uint32_t ko = (uint32_t)st * 128u;
      const bool live = st < n_st;
      if (u == 0)
        set_m0(g == 0 ? lds_a + (uint32_t)sl * SLOT_A
                      : lds_b + (uint32_t)sl * SLOT_B + (uint32_t)(g - 1) * 4096u);
      const uint32_t voff = g == 0 ? a_off + (uint32_t)u * a8
                                   : b_off + (uint32_t)(4 * (g - 1) + u) * b8;
      if (g == 0 || !NT) {
        const i32x4 d = desc_at(g == 0 ? da : dbw, ko, live);
        switch (u) {
          case 0: lds_dma16_m0<0>(d, voff); break;
          case 1: lds_dma16_m0<1024>(d, voff - 1024u); break;
          case 2: lds_dma16_m0<2048>(d, voff - 2048u); break;
          default: lds_dma16_m0<3072>(d, voff - 3072u); break;
        }
      } else {
        const i32x4 d = desc_at(dbw, ko, live);
        switch (u) {
          case 0: lds_dma16_m0_nt<0>(d, voff); break;
          case 1: lds_dma16_m0_nt<1024>(d, voff - 1024u); break;
          case 2: lds_dma16_m0_nt<2048>(d, voff - 2048u); break;
          default: lds_dma16_m0_nt<3072>(d, voff - 3072u); break;
        }
      }
    };
    const int ri = lane & 15, rg = lane >> 4;
    const int fa0 = ri * 8, fb0 = (64 * wave + ri) * 8;
    const int fs0 = rg ^ (ri & 7), fs1 = (4 + rg) ^ (ri & 7);
    // the 12 fragments of a half: B (4) in calls 0-1, A (8) in calls 2-5
    auto read_set = [&](int i, const i32x4* pa, const i32x4* pb, int fs, i32x4 (&fa)[8],
                        i32x4 (&fb)[4]) {
      if (i < 2) {
        fb[2 * i] = pb[fb0 + 128 * (2 * i) + fs];
        fb[2 * i + 1] = pb[fb0 + 128 * (2 * i + 1) + fs];
      } else if (i < 6) {
        fa[2 * i - 4] = pa[fa0 + 128 * (2 * i - 4) + fs];
        fa[2 * i - 3] = pa[fa0 + 128 * (2 * i - 3) + fs];
      }
    };
    auto mma_row = [&](int i, const i32x4 (&fa)[8], const i32x4 (&fb)[4]) {
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = mma16(Tag{}, fa[i], fb[j], acc[i][j]);
    };
    i32x4 h0a[8], h0b[4], h1a[8], h1b[4];

    // prologue: stages 0 and 1 on their way, stage 0 landed, stage 2 issued
    // into the third slot, h0 of stage 0 in registers
#pragma unroll
    for (int n = 0; n < 12; ++n) issue(0, 0, n);
#pragma unroll
    for (int n = 0; n < 12; ++n) issue(1, 1, n);
    gemm_wait_vm<12>();
    __builtin_amdgcn_s_barrier();
#pragma unroll
    for (int n = 0; n < 12; ++n) issue(2, 2, n);
    {
      const i32x4* pa = sm.a[0];
      const i32x4* pb = sm.b[0];
#pragma unroll
      for (int i = 0; i < 8; ++i) h0a[i] = pa[fa0 + 128 * i + fs0];
#pragma unroll
      for (int j = 0; j < 4; ++j) h0b[j] = pb[fb0 + 128 * j + fs0];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        read_set(i, pa, pb, fs1, h1a, h1b);
        __builtin_amdgcn_sched_barrier(0);
        mma_row(i, h0a, h0b);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    int sl = 1;  // slot of stage st
    for (int st = 1; st < n_st; ++st) {
      // stage st landed (stage st + 1's loads may still be in flight); this
      // wave's reads of stage st - 1 are complete
      gemm_wait_vm<12>();
      wait_lgkm0();
      __builtin_amdgcn_s_barrier();
      const int sl2 = sl == 0 ? 2 : sl - 1;  // slot of stage st - 1 = slot of st + 2
      const i32x4* pa = sm.a[sl];
      const i32x4* pb = sm.b[sl];
      // h1 of stage st - 1, reading h0 of stage st, loading stage st + 2
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        read_set(i, pa, pb, fs0, h0a, h0b);
        if (2 * i < 12) issue(st + 2, sl2, 2 * i);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = mma16(Tag{}, h1a[i], h1b[j], acc[i][j]);
        __builtin_amdgcn_sched_barrier(0);
        if (2 * i + 1 < 12) issue(st + 2, sl2, 2 * i + 1);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int j = 2; j < 4; ++j) acc[i][j] = mma16(Tag{}, h1a[i], h1b[j], acc[i][j]);
        __builtin_amdgcn_sched_barrier(0);
      }
      // h0 of stage st, reading h1 of stage st
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        read_set(i, pa, pb, fs1, h1a, h1b);
        __builtin_amdgcn_sched_barrier(0);
        mma_row(i, h0a, h0b);
        __builtin_amdgcn_sched_barrier(0);
      }
      sl = sl == 2 ? 0 : sl + 1;
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) mma_row(i, h1a, h1b);
    // the zero-filling loads past the end have landed and every wave's LDS
    // reads are complete before the workgroup moves on
    gemm_wait_vm<0>();
    wait_lgkm0();
    __builtin_amdgcn_s_barrier();
  }

  static constexpr int NJ = 4;  // 16-column accumulator blocks per wave
  __device__ static inline int row_of(int i, int r) {
    const int lane = threadIdx.x & 63;
    return 16 * i + 4 * (lane >> 4) + r;
  }
  __device__ static inline int col_of(int j) {
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    return 64 * wave + 16 * j + (lane & 15);
  }
  __device__ static inline int col_base() { return 64 * (int)(threadIdx.x >> 6); }
};

// The same block tile for K-major operands: C[m][n] += sum_k AT[k][m] BT[k][n]
// with K-rows of the tile's 256 contiguous columns (A: rows of AT from the
// tile's first column; B likewise; both with the row stride ld).  A stage is 64 K-rows of
// 512 bytes per operand, loaded by the same direct-to-LDS instructions (two
// K-rows per instruction); in LDS the 32-byte piece P of K-row r sits at
// P ^ g(r), g(r) = (r & 3) | ((r >> 3) & 1) << 2, so that the 16 K-rows one
// fragment read touches fall into distinct banks.  Fragments are read with
// ds_read_b64_tr_b16, which transposes 4 x 16 blocks of 16-bit values within
// each 16-lane group: lane i of group rg receives column i of four
// consecutive K-rows; two such reads give the 8 K-values of an MFMA operand.
// It issues twice as many LDS reads as the row-major core (512 instead of
// 1024 bytes each) and needs no transposed copy of the operands.
//
// NEG: the sign bit of every 16-bit value of the B fragments is flipped (XOR
// 0x80008000, in place: flip_sign16) between the loop that reads a K-half
// and the loop that uses it, so the core accumulates -A B^T.  The
// second-moment accumulation alternates the sign of its row slices this way to cancel the matrix core's rounding bias (see
// syrk.hip).  It is a compile-time choice: the non-negated core is the
// plain loop, and a run-time mask or branch inside the loop raised the
// scalar-register pressure or the instruction count of every slice.
typedef short s16x4 __attribute__((ext_vector_type(4)));
__device__ inline i32x2 lds_read_tr16(uint32_t byte_addr) {
  const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) s16x4*)(uintptr_t)byte_addr);
  return __builtin_bit_cast(i32x2, v);
}
__device__ inline int kmajor_swz(int r) { return (r & 3) | (((r >> 3) & 1) << 2); }

// Flip the sign of the eight 16-bit values of an MFMA operand fragment, in
// its own registers.  Written as plain code, the flipped values got fresh
// registers, and in the negated core's paired stage loop the register file
// ran short and the compiler moved accumulators in and out of it; inline
// asm keeps them in place.  The asm is opaque to the compiler's hazard
// checks, so a block of flips ends with s_nop 4 (five wait states; a VALU
// write of a VGPR needs two before an MFMA reads it), and the build scans
// the assembly for an MFMA that reads a flipped register too soon.
__device__ inline void flip_sign16(i32x4& f) {
  asm volatile("v_xor_b32 %0, 0x80008000, %0" : "+v"(f.x));
  asm volatile("v_xor_b32 %0, 0x80008000, %0" : "+v"(f.y));
  asm volatile("v_xor_b32 %0, 0x80008000, %0" : "+v"(f.z));
  asm volatile("v_xor_b32 %0, 0x80008000, %0" : "+v"(f.w));
}

template <typename Tag, bool NEG = false>
struct GemmCoreT {
  f32x4 acc[8][8];

  __device__ inline void zero() {
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // n_st stages of 64 K-rows; K-rows past a descriptor's range read zeros.
  // Byte offsets within a descriptor must fit 31 bits.
  __device__ inline void run(GemmSmem& sm, const i32x4& da, const i32x4& db, int64_t ld,
                             int n_st) {
    if (n_st <= 0) return;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int lane = threadIdx.x & 63;
    const int wm = wave >> 1, wn = wave & 1;
    // loads: instruction h (0..7) of a wave covers K-rows 16 wave + 2 h +
    // lane / 32; the lane's LDS chunk s = lane % 32 receives global chunk
    // ((s / 2) ^ g(row)) * 2 + s % 2; offsets carry -1024 (h % 4) for the
    // instruction offset that places four loads behind one M0 write
    const int lr = lane >> 5, s = lane & 31;
    uint32_t oa[8];
#pragma unroll
    for (int h = 0; h < 8; ++h) {
      const int row = 16 * wave + 2 * h + lr;
      const int c = (((s >> 1) ^ kmajor_swz(row)) << 1) | (s & 1);
      oa[h] = (uint32_t)((int64_t)row * ld * 2 + c * 16) - 1024u * (uint32_t)(h & 3);
    }
    const uint32_t kst = (uint32_t)(64 * ld * 2);
    const uint32_t sa0 = (uint32_t)(uintptr_t)&sm.a[0][0], sb0 = (uint32_t)(uintptr_t)&sm.b[0][0];
    const uint32_t lds_a = sa0 + (uint32_t)(16 * wave) * 512u;
    const uint32_t lds_b = sb0 + (uint32_t)(16 * wave) * 512u;
    auto issue_grp = [&](int st, int g) {
      const uint32_t sb = (uint32_t)(st & 1) * G_SLOT;
      set_m0((g < 2 ? lds_a : lds_b) + sb + (uint32_t)(g & 1) * 4096u);
    };
    // the same for a stage whose slot is known at compile time
    auto issue_grp_s = [&](auto slot_c, int g) {
      constexpr uint32_t sb = (uint32_t)decltype(slot_c)::value * G_SLOT;
      set_m0((g < 2 ? lds_a : lds_b) + sb + (uint32_t)(g & 1) * 4096u);
    };
    auto issue_u = [&](int st, int g, auto uc) {
      constexpr int u = decltype(uc)::value;
      const bool live = st < n_st;
      const int h = 4 * (g & 1) + u;
      if (g < 2) {
        lds_dma16_m0<1024 * u>(desc_at(da, (uint32_t)st * kst, live), oa[h]);
      } else {
        lds_dma16_m0<1024 * u>(desc_at(db, (uint32_t)st * kst, live), oa[h]);
      }
    };
    auto issue_all = [&](int st) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        issue_grp(st, g);
        issue_u(st, g, std::integral_constant<int, 0>{});
        issue_u(st, g, std::integral_constant<int, 1>{});
        issue_u(st, g, std::integral_constant<int, 2>{});
        issue_u(st, g, std::integral_constant<int, 3>{});
      }
    };
    // fragment of 16-column block t (of the wave's 128) in K-half hk: lane
    // (rg, i) reads K-rows 32 hk + 8 rg + 4 h + i / 4 (h = 0, 1), columns
    // 16 t + 4 (i % 4) .. + 3 of its operand half wx.  The lane's address
    // of block t in slot 0, K-half 0 is fixed (fpa, fpb); the slot and the
    // K-half add a constant that the reads carry in their offset field (the
    // stage loop runs in pairs, so every stage's slot is known at compile
    // time), and no address arithmetic is left in the loop.
    const int rg = lane >> 4, i4 = lane & 15;
    const int gl = (i4 >> 2) | ((rg & 1) << 2);  // g() of every K-row this lane reads
    const uint32_t rowb = (uint32_t)(8 * rg + (i4 >> 2)) * 512u + 8u * (uint32_t)(i4 & 3);
    uint32_t fpa[8], fpb[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      fpa[t] = sa0 + rowb + 32u * (uint32_t)((8 * wm + t) ^ gl);
      fpb[t] = sb0 + rowb + 32u * (uint32_t)((8 * wn + t) ^ gl);
    }
    auto frag = [&](uint32_t addr) -> i32x4 {
      const i32x2 lo = lds_read_tr16(addr);
      const i32x2 hi = lds_read_tr16(addr + 4u * 512u);
      return i32x4{lo.x, lo.y, hi.x, hi.y};
    };
    // the 16 fragments of a half (slot and K-half in off), two per call, B
    // first (as in GemmCore)
    auto read_pair = [&](int i, uint32_t off, i32x4 (&fa)[8], i32x4 (&fb)[8]) {
      if (i < 4) {
        fb[2 * i] = frag(fpb[2 * i] + off);
        fb[2 * i + 1] = frag(fpb[2 * i + 1] + off);
      } else {
        fa[2 * i - 8] = frag(fpa[2 * i - 8] + off);
        fa[2 * i - 7] = frag(fpa[2 * i - 7] + off);
      }
    };
    auto mma_row = [&](int i, const i32x4 (&fa)[8], const i32x4 (&fb)[8]) {
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[i][j] = mma16(Tag{}, fa[i], fb[j], acc[i][j]);
    };
    // NEG: the B fragments of a K-half are flipped in place once their reads
    // have landed, between the loop that read them and the loop that uses
    // them
    auto negate_b = [&](i32x4 (&fb)[8]) {
      if (NEG) {
#pragma unroll
        for (int j = 0; j < 8; ++j) flip_sign16(fb[j]);
        asm volatile("s_nop 4");
      }
    };
    i32x4 h0a[8], h0b[8], h1a[8], h1b[8];

    // same pipeline as GemmCore::run
    constexpr uint32_t HK1 = 32u * 512u;  // K-half 1 of a slot
    issue_all(0);
    gemm_wait_vm<0>();
    __builtin_amdgcn_s_barrier();
    issue_all(1);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      h0a[i] = frag(fpa[i]);
      h0b[i] = frag(fpb[i]);
    }
    negate_b(h0b);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      read_pair(i, HK1, h1a, h1b);
      __builtin_amdgcn_sched_barrier(0);
      mma_row(i, h0a, h0b);
      __builtin_amdgcn_sched_barrier(0);
    }
    negate_b(h1b);
    // stage st in slot SLOT = st & 1 (a compile-time constant)
    auto stage = [&](int st, auto slot_c) {
      constexpr uint32_t SLOT = decltype(slot_c)::value;
      constexpr uint32_t base = SLOT * G_SLOT;
      gemm_wait_vm<0>();
      wait_lgkm0();
      __builtin_amdgcn_s_barrier();
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        read_pair(i, base, h0a, h0b);
        if ((i & 1) == 0) {
          issue_grp_s(std::integral_constant<uint32_t, 1u - SLOT>{}, i >> 1);
          issue_u(st + 1, i >> 1, std::integral_constant<int, 0>{});
        } else {
          issue_u(st + 1, i >> 1, std::integral_constant<int, 2>{});
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = mma16(Tag{}, h1a[i], h1b[j], acc[i][j]);
        __builtin_amdgcn_sched_barrier(0);
        if ((i & 1) == 0) {
          issue_u(st + 1, i >> 1, std::integral_constant<int, 1>{});
        } else {
          issue_u(st + 1, i >> 1, std::integral_constant<int, 3>{});
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int j = 4; j < 8; ++j) acc[i][j] = mma16(Tag{}, h1a[i], h1b[j], acc[i][j]);
        __builtin_amdgcn_sched_barrier(0);
      }
      negate_b(h0b);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        read_pair(i, base + HK1, h1a, h1b);
        __builtin_amdgcn_sched_barrier(0);
        mma_row(i, h0a, h0b);
        __builtin_amdgcn_sched_barrier(0);
      }
      negate_b(h1b);
    };
    int st = 1;
    for (; st + 1 < n_st; st += 2) {
      stage(st, std::integral_constant<uint32_t, 1>{});
      stage(st + 1, std::integral_constant<uint32_t, 0>{});
    }
    if (st < n_st) stage(st, std::integral_constant<uint32_t, 1>{});
#pragma unroll
    for (int i = 0; i < 8; ++i) mma_row(i, h1a, h1b);
    gemm_wait_vm<0>();
    wait_lgkm0();
    __builtin_amdgcn_s_barrier();
  }
};

}  // namespace attr
