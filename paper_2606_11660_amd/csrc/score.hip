// Query x gradient-store scoring with exact streaming top-k (section
// "Attribution Pipelines": every gradient store supports exact top-k lookup
// of the most influential items).
//
// Score tiles are 64 queries x 128 store rows, a matrix-core GEMM over D
// (fp16 16x16x32 or fp32 16x16x4 MFMA, fp32 accumulate).  Store rows stream
// with line-coalesced loads and pass through a per-wave LDS tile into MFMA
// fragments (as in the projection); query fragments come from L2.
//
// Three plans, chosen on the host from the problem shape:
//  * streaming (large stores, fewer than 128 fp16 queries): see
//    score_stream_kernel.  Rows are visited in increasing index order, so a
//    strict ">" keeps the lower index on ties.  The Q x N score matrix never
//    reaches memory.
//  * GEMM (128 or more fp16 queries): the 256 x 256 GEMM core scores chunks
//    of rows into the workspace and an exact selection kernel reads them.
//  * split-K (small stores, too few tiles to fill 256 CUs): workgroups own
//    (tile, D-slice) pairs and write fp32 partial scores; one workgroup per
//    query and part of the rows sums the slices in slice order and selects
//    by a threshold from 16-row segment maxima and a sort.
// Either way, per-partition sorted lists are merged per query by block-wide
// arg-max in (score desc, index asc) order, which also merges a previous
// result when a store is scored chunk by chunk.
#include "common.h"
#include "gemm.h"
#include "kernels.h"

namespace attr {
namespace {

constexpr int SQB = 64;       // queries per workgroup
constexpr int STN = 128;      // store rows per tile (4 waves x 32 rows)
constexpr int SPD = 3;        // 128-byte K-groups of store loads in flight (5 or 7: no faster)

template <bool F16>
struct STag;
template <>
struct STag<true> {
  using tag = F16Tag;
  static constexpr int bytes = 2;
};
template <>
struct STag<false> {
  using tag = F32Tag;
  static constexpr int bytes = 4;
};

// acc[qt][rt] (+)= Q[16 qt + i, groups) . G[32 wave + 16 rt + j, groups) for
// the K-groups [g_begin, g_end).  Lane layout of acc: query 16 qt + 4 (lane
// / 16) + r (register r), row 16 rt + lane % 16.
template <bool F16>
__device__ inline void score_tile(__amdgpu_buffer_rsrc_t rq, int64_t ldq,
                                  __amdgpu_buffer_rsrc_t rg, int64_t ldg, int g_begin,
                                  int g_end, int lane, i32x4* __restrict__ xp,
                                  f32x4 (&acc)[4][2]) {
  using Tag = typename STag<F16>::tag;
  constexpr int EB = STag<F16>::bytes;
  constexpr int E = 16 / EB;
  constexpr int KS = 4 * E;
  const int lrow = lane >> 3, lch = lane & 7;
  const uint32_t g_base = (uint32_t)((int64_t)lrow * ldg * EB + lch * 16);
  const uint32_t g_half = (uint32_t)(8 * ldg * EB);
  const uint32_t g_tile = (uint32_t)(16 * ldg * EB);
  const int wslot = lrow * 8 + (lch ^ lrow);
  const int ri = lane & 15, rgrp = lane >> 4;
  const int rslot0 = ri * 8 + (rgrp ^ (ri & 7));
  const int rslot1 = ri * 8 + ((4 + rgrp) ^ (ri & 7));
  const uint32_t q_base = (uint32_t)(((int64_t)ri * ldq + E * rgrp) * EB);
  const uint32_t q_tile = (uint32_t)(16 * ldq * EB);

  i32x4 gbuf[SPD][2][2], qcur[2][4], qnxt[2][4];
  auto issue_g = [&](int grp, i32x4 (&gb)[2][2]) {
    const uint32_t off = g_base + (uint32_t)grp * 128u;
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      gb[rt][0] = load16_stream(rg, off + rt * g_tile);
      gb[rt][1] = load16_stream(rg, off + rt * g_tile + g_half);
    }
  };
  auto issue_q = [&](int grp, i32x4 (&qf)[2][4]) {
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int qt = 0; qt < 4; ++qt)
        qf[s][qt] = load16_cached(rq, q_base + qt * q_tile + (uint32_t)((2 * grp + s) * KS * EB));
  };
#pragma unroll
  for (int u = 0; u < SPD - 1; ++u)
    if (g_begin + u < g_end) issue_g(g_begin + u, gbuf[u]);
  issue_q(g_begin, qcur);

  for (int g0 = g_begin; g0 < g_end; g0 += SPD) {
#pragma unroll
    for (int u = 0; u < SPD; ++u) {
      const int grp = g0 + u;
      if (grp + SPD - 1 < g_end) issue_g(grp + SPD - 1, gbuf[(u + SPD - 1) % SPD]);
      if (grp < g_end) {
        if (grp + 1 < g_end) issue_q(grp + 1, qnxt);
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) {
          xp[rt * 128 + wslot] = gbuf[u][rt][0];
          xp[rt * 128 + 64 + wslot] = gbuf[u][rt][1];
        }
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) {
          const i32x4 f0 = xp[rt * 128 + rslot0];
          const i32x4 f1 = xp[rt * 128 + rslot1];
#pragma unroll
          for (int qt = 0; qt < 4; ++qt) {
            acc[qt][rt] = mma16(Tag{}, qcur[0][qt], f0, acc[qt][rt]);
            acc[qt][rt] = mma16(Tag{}, qcur[1][qt], f1, acc[qt][rt]);
          }
        }
#pragma unroll
        for (int s = 0; s < 2; ++s)
#pragma unroll
          for (int qt = 0; qt < 4; ++qt) qcur[s][qt] = qnxt[s][qt];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// streaming plan (large stores)
// ---------------------------------------------------------------------------
// A workgroup owns 64 queries (16 per wave) and a contiguous partition of
// store rows, walked in tiles of 64 TR rows (TR = 1 or 2).  The tile
// sequence is cut into 128-byte K-groups ("stages"): for every stage the
// tile's store rows and the 64 query rows go straight from memory into a
// shared LDS ring by
// direct-to-LDS buffer loads (1 KB, line-coalesced instructions that land in
// the XOR-swizzled fragment layout), RING - 1 stages ahead.  No vector load
// feeds a register inside the loop, so the only waits are explicit: every
// stage costs each wave exactly LPW = 2 (TR + 1) load instructions, the wait
// for stage st is vmcnt <= LPW * (stages issued after st), then one barrier
// (all waves' loads landed; all waves finished the previous stage, whose
// slot is then refilled).
//
// Each wave computes its 16 queries (every fourth of the block) x the tile,
// so after a tile it holds every score of its own queries and needs no
// exchange.  Top-k selection is software-pipelined behind the stream: when
// a tile ends its scores move to a pending copy and are compared with the
// 16 running thresholds (k-th best so far, kept in registers); during the
// next tile's stages the wave walks its queries in order, a few per stage,
// and inserts the passing rows of each, in row order.  Each query's sorted
// list is held in registers (entry p in lane p % 64 of register p / 64,
// padded with (-inf, -1)); an insertion uses all 64 lanes at once (the
// position is the number of entries >= s: existing entries have lower row
// indices, so ties keep them first; the tail moves one lane up through a
// wave-wide DPP shift).  Register arrays need compile-time indices, so the
// query being served is always list 0 and the wave's list array rotates by
// one after each query (16 moves of one or two registers pairs): the
// selection code is one short loop body, not a per-query unrolled copy,
// and it stays in the instruction cache.
//
// Optionally each query starts from a floor: a lower bound on its k-th best
// score over the whole store.  Rows below the floor cannot be in the
// answer, so they never enter a list; without it every partition list fills
// with k rows and then takes ~k ln(rows / k) more insertions, which at 64
// queries and k = 100 cost more than the stream itself.  The bound is the
// k-th largest of the maxima of the first 16384 rows' 64-row segments (k
// distinct rows score at least that much), found by this kernel run with
// k = 1 over one-tile partitions and a per-query sort of the 256 maxima.
// A list then may end with fewer than k rows above the floor; the merge
// takes the global top k, all of which are at or above it.
// Partitions are mapped so that the query blocks sharing a partition run on
// the same XCD at the same time and share its L2.
constexpr int SR = 64;  // store rows per tile
constexpr int SQ = 64;  // queries per workgroup

template <int N>
__device__ inline void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
// vmcnt <= n for a run-time n that is a multiple of L (n <= 6 L)
template <int L>
__device__ inline void wait_vmcnt_m(int n) {
  switch (n / L) {
    case 6: wait_vmcnt<6 * L>(); break;
    case 5: wait_vmcnt<5 * L>(); break;
    case 4: wait_vmcnt<4 * L>(); break;
    case 3: wait_vmcnt<3 * L>(); break;
    case 2: wait_vmcnt<2 * L>(); break;
    case 1: wait_vmcnt<L>(); break;
    default: wait_vmcnt<0>(); break;
  }
}

__device__ inline float sel4(const f32x4& a, int r) {
  float v = a[0];
  v = r == 1 ? a[1] : v;
  v = r == 2 ? a[2] : v;
  v = r == 3 ? a[3] : v;
  return v;
}

// lane l takes lane l - 1's value, lane 0 takes `fill` (DPP wave_shr:1)
__device__ inline int wave_shr1(int v, int fill) {
  return __builtin_amdgcn_update_dpp(fill, v, 0x138, 0xf, 0xf, false);
}

// Largest float below x (-inf for x = -inf or NaN): a strict ">" against it
// admits every score >= x.
__device__ inline float float_below(float x) {
  if (!(x > -__builtin_inff())) return -__builtin_inff();
  if (x == 0.f) return -__builtin_bit_cast(float, 1);  // -denorm_min
  const int b = __builtin_bit_cast(int, x);
  return __builtin_bit_cast(float, x > 0.f ? b - 1 : b + 1);  // +inf -> FLT_MAX
}

// Register-resident sorted list of one query: entry p in lane p % 64 of
// slot p / 64; positions >= k are don't-care.
template <int NS>
struct RegList {
  float s[NS];
  int i[NS];
  // kth entry's score
  __device__ inline float kth(int k) const {
    float t = s[0];
#pragma unroll
    for (int j = 1; j < NS; ++j) t = (k - 1) / 64 == j ? s[j] : t;
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, t), (k - 1) & 63));
  }
  // insert (v, idx): idx exceeds every row present, v > kth(k)
  __device__ inline void insert(float v, int idx, int k, int lane) {
    int pos = 0;
#pragma unroll
    for (int j = 0; j < NS; ++j)
      pos += __builtin_popcountll(__builtin_amdgcn_ballot_w64(64 * j + lane < k && s[j] >= v));
    float us[NS];
    int ui[NS];
#pragma unroll
    for (int j = 0; j < NS; ++j) {
      const int cs = j ? __builtin_amdgcn_readlane(__builtin_bit_cast(int, s[j - 1]), 63) : 0;
      const int ci = j ? __builtin_amdgcn_readlane(i[j - 1], 63) : 0;
      us[j] = __builtin_bit_cast(float, wave_shr1(__builtin_bit_cast(int, s[j]), cs));
      ui[j] = wave_shr1(i[j], ci);
    }
#pragma unroll
    for (int j = 0; j < NS; ++j) {
      const int p = 64 * j + lane;
      s[j] = p < pos ? s[j] : (p == pos ? v : us[j]);
      i[j] = p < pos ? i[j] : (p == pos ? idx : ui[j]);
    }
  }
};

// At least two waves per SIMD (two workgroups per CU): the compiler keeps
// every configuration within 256 VGPRs (64 queries with two-register lists
// and 128-row tiles would otherwise take 268 and run one workgroup per CU).
template <bool F16, int KMAX, int RING, int GPS, int QPW, int TR>
__global__ __launch_bounds__(256, 2) void score_stream_kernel(
    const char* __restrict__ Q, int64_t n_q, int64_t ldq, const char* __restrict__ G,
    int64_t n_g, int64_t ldg, int n_grp, int k, int64_t rows_per_part, int n_parts, int n_qb,
    const float* __restrict__ bound, float* __restrict__ part_s, int64_t* __restrict__ part_i,
    int64_t index_base) {
  // GPS 128-byte K-groups per stage: a stage row is RB bytes (CPR chunks),
  // RPI rows per 1 KB load; tiles of SRT = 64 TR store rows; LPW loads per
  // wave and stage (16 TR store rows and 16 query rows)
  constexpr int SRT = SR * TR;
  constexpr int RB = 128 * GPS, CPR = 8 * GPS, RPI = 8 / GPS, LPW = 2 * GPS * (TR + 1);
  static_assert(RING >= 3 && RING - 2 <= 6, "wait_vmcnt_m range");
  static_assert(TR == 1 || TR == 2, "candidate bits: 4 TR row tiles x 4 queries");
  using Tag = typename STag<F16>::tag;
  constexpr int EB = STag<F16>::bytes;
  constexpr int NS = (KMAX + 63) / 64;
  __shared__ i32x4 ring[RING][(SRT + SQ) * CPR];  // store rows, then query rows

  const uint32_t b = blockIdx.x;
  const int xcd = (int)(b & 7u);
  const uint32_t jb = b >> 3;
  const int qb = (int)(jb % (uint32_t)n_qb);
  const int p = (int)(jb / (uint32_t)n_qb) * 8 + xcd;
  if (p >= n_parts) return;  // uniform
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int lane = threadIdx.x & 63;

  const int64_t q0 = (int64_t)qb * SQ;
  int64_t nq_blk = n_q - q0;
  nq_blk = nq_blk > SQ ? SQ : nq_blk;
  // wave w holds block queries w, w + 4, ..., w + 60 (slot j = query 4 j + w), so
  // that a partial block spreads its selection work over all four waves
  int nq_w = (int)((nq_blk - wave + 3) / 4);
  nq_w = nq_w < 0 ? 0 : (nq_w > QPW ? QPW : nq_w);  // the host sizes QPW to the block
  // a store read by a single query block is not kept in L2
  const bool g_nt = n_qb == 1;

  const int64_t r_begin = (int64_t)p * rows_per_part;
  int64_t r_end = r_begin + rows_per_part;
  r_end = r_end > n_g ? n_g : r_end;
  const int64_t nrows = r_end > r_begin ? r_end - r_begin : 0;
  const int n_tiles = (int)((nrows + SRT - 1) / SRT);
  const int n_stg = n_grp / GPS;  // stages per tile (n_grp is a multiple of GPS)
  const int total = n_tiles * n_stg;
  const int spg = (QPW + n_stg - 1) / n_stg;  // selection steps per stage

  // the wave's QPW sorted lists, in registers; the list of the query being
  // selected is always lists[0]: the array rotates by one after every step
  RegList<NS> lists[QPW];
#pragma unroll
  for (int ql = 0; ql < QPW; ++ql)
#pragma unroll
    for (int j = 0; j < NS; ++j) {
      lists[ql].s[j] = -__builtin_inff();
      lists[ql].i[j] = -1;
    }
  auto rotate = [&]() {
    const RegList<NS> t = lists[0];
#pragma unroll
    for (int ql = 0; ql + 1 < QPW; ++ql) lists[ql] = lists[ql + 1];
    lists[QPW - 1] = t;
  };

  const i32x4 dq = make_desc(Q + q0 * ldq * EB, (uint32_t)(nq_blk * ldq * EB));
  // load lane -> row lr of the instruction's RPI rows, LDS slot lane % CPR of
  // that row, which holds chunk (lane % CPR) ^ (row % 8)
  const int lr = lane / CPR;
  const int ri = lane & 15, rgrp = lane >> 4;
  const uint32_t ring_base = (uint32_t)(uintptr_t)&ring[0][0];
  constexpr uint32_t SLOT_BYTES = (SRT + SQ) * RB;
  // per-lane byte offsets of this wave's 16 TR store rows / 16 query rows in
  // groups of RPI rows (stage 0); query slot j is block query 4 j + wave
  uint32_t goff[2 * GPS * TR], qoff[2 * GPS];
#pragma unroll
  for (int h = 0; h < 2 * GPS * TR; ++h) {
    const int lc = (lane % CPR) ^ ((RPI * h + lr) & 7);  // LDS rows 16 TR wave + RPI h + lr
    goff[h] = (uint32_t)((int64_t)(16 * TR * wave + RPI * h + lr) * ldg * EB + lc * 16);
  }
#pragma unroll
  for (int h = 0; h < 2 * GPS; ++h) {
    const int lc = (lane % CPR) ^ ((RPI * h + lr) & 7);  // LDS rows SRT + 16 wave + RPI h + lr
    qoff[h] = (uint32_t)((int64_t)(4 * (RPI * h + lr) + wave) * ldq * EB + lc * 16);
  }
  const uint32_t lds_g = ring_base + (uint32_t)(16 * TR * wave) * RB;
  const uint32_t lds_q = ring_base + (uint32_t)(SRT + 16 * wave) * RB;

  // issue cursor: next stage to load is (it_tile, it_g) into slot islot
  int it_tile = 0, it_g = 0, issued = 0, islot = 0;
  i32x4 dt{0, 0, 0, 0};
  auto tile_desc = [&](int tile) {
    const int64_t row0 = r_begin + (int64_t)tile * SRT;
    int64_t nr = r_end - row0;
    nr = nr > SRT ? SRT : nr;
    dt = make_desc(G + row0 * ldg * EB, (uint32_t)(nr * ldg * EB));
  };
  auto issue_next = [&]() {
    const uint32_t sb = (uint32_t)islot * SLOT_BYTES;
    const uint32_t go = (uint32_t)it_g * RB;
    if (g_nt) {
#pragma unroll
      for (int h = 0; h < 2 * GPS * TR; ++h) lds_dma16_nt(dt, goff[h] + go, lds_g + sb + 1024u * h);
    } else {
#pragma unroll
      for (int h = 0; h < 2 * GPS * TR; ++h) lds_dma16(dt, goff[h] + go, lds_g + sb + 1024u * h);
    }
#pragma unroll
    for (int h = 0; h < 2 * GPS; ++h) lds_dma16(dq, qoff[h] + go, lds_q + sb + 1024u * h);
    ++issued;
    islot = islot == RING - 1 ? 0 : islot + 1;
    if (++it_g == n_stg) {
      it_g = 0;
      ++it_tile;
      if (it_tile < n_tiles) tile_desc(it_tile);
    }
  };

  if (total > 0) tile_desc(0);
#pragma unroll
  for (int u = 0; u < RING - 1; ++u)
    if (issued < total) issue_next();

  // floor4: per query, the largest float below a lower bound on its k-th
  // best score over the whole store (rows below it cannot be in the answer),
  // else -inf; running thresholds thr4 start there.  Lane l of thr4[r] and
  // floor4[r] holds slot 4 (l / 16) + r.
  f32x4 floor4 = f32x4{-__builtin_inff(), -__builtin_inff(), -__builtin_inff(), -__builtin_inff()};
  if (bound) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int ql = 4 * rgrp + r;
      if (ql < nq_w) floor4[r] = float_below(bound[q0 + 4 * ql + wave]);
    }
  }
  f32x4 thr4 = floor4;
  // pending tile: scores (pend[rt][r] in lane l: query 4 (l / 16) + r, row
  // 16 rt + l % 16), candidate bits cm (bit 4 rt + r) and its first row
  f32x4 pend[4 * TR];
  uint32_t cm = 0;
  bool pend_any = false;
  int pend_rbase = 0;

  auto process_query = [&](int ql, RegList<NS>& L) {
    const int r = ql & 3, grp = ql >> 2;
    uint64_t m[4 * TR];
    bool has = false;
#pragma unroll
    for (int rt = 0; rt < 4 * TR; ++rt) {
      m[rt] = __builtin_amdgcn_ballot_w64(rgrp == grp && ((cm >> (4 * rt + r)) & 1u));
      has |= m[rt] != 0;
    }
    if (!has) return;
    float thr = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, sel4(thr4, r)), 16 * grp));
    const float flo = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, sel4(floor4, r)), 16 * grp));
#pragma unroll
    for (int rt = 0; rt < 4 * TR; ++rt) {
      const float v = sel4(pend[rt], r);
      uint64_t mm = m[rt];
      while (mm) {
        const int src = __builtin_ctzll(mm);
        mm &= mm - 1;
        const float cv = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), src));
        if (cv > thr) {
          L.insert(cv, pend_rbase + 16 * rt + (src & 15), k, lane);
          thr = fmaxf(L.kth(k), flo);
        }
      }
    }
    const bool mine = rgrp == grp;
    thr4[0] = mine && r == 0 ? thr : thr4[0];
    thr4[1] = mine && r == 1 ? thr : thr4[1];
    thr4[2] = mine && r == 2 ? thr : thr4[2];
    thr4[3] = mine && r == 3 ? thr : thr4[3];
  };

  int st = 0, cslot = 0;
  for (int tile = 0; tile < n_tiles; ++tile) {
    f32x4 acc[4 * TR];
#pragma unroll
    for (int rt = 0; rt < 4 * TR; ++rt) acc[rt] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int g = 0; g < n_stg; ++g, ++st) {
      // stage st landed: at most (loads issued after it) of this wave's
      // loads are still outstanding
      const int after = total - 1 - st;
      if (after >= RING - 2) {
        wait_vmcnt<LPW * (RING - 2)>();
      } else {
        wait_vmcnt_m<LPW>(LPW * after);
      }
      // this wave's LDS reads of the previous stage are complete before
      // anyone refills that slot
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      __builtin_amdgcn_s_barrier();
      if (issued < total) issue_next();
      const i32x4* sl = ring[cslot];
      cslot = cslot == RING - 1 ? 0 : cslot + 1;
#pragma unroll
      for (int s2 = 0; s2 < 2 * GPS; ++s2) {
        const int qrow = SRT + 16 * wave + ri;
        const i32x4 qf = sl[qrow * CPR + ((4 * s2 + rgrp) ^ (qrow & 7))];
#pragma unroll
        for (int rt = 0; rt < 4 * TR; ++rt) {
          const int grow = 16 * rt + ri;
          const i32x4 gf = sl[grow * CPR + ((4 * s2 + rgrp) ^ (grow & 7))];
          acc[rt] = mma16(Tag{}, qf, gf, acc[rt]);
        }
      }
      // previous tile's selection, spread over this tile's stages
      // steps [g c, (g + 1) c) of the QPW, in order, c = ceil(QPW / n_stg)
      if (pend_any)
        for (int ql = g * spg; ql < QPW && ql < (g + 1) * spg; ++ql) {
          if (ql < nq_w) process_query(ql, lists[0]);
          rotate();
        }
    }
    // hand this tile over to the selection
    const int rbase = tile * SRT;
    const int nvalid = (int)(nrows - rbase > SRT ? SRT : nrows - rbase);
    cm = 0;
#pragma unroll
    for (int rt = 0; rt < 4 * TR; ++rt) {
      pend[rt] = acc[rt];
#pragma unroll
      for (int r = 0; r < 4; ++r)
        cm |= (4 * rgrp + r < nq_w && 16 * rt + ri < nvalid && acc[rt][r] > thr4[r]) ? 1u << (4 * rt + r) : 0u;
    }
    pend_any = __builtin_amdgcn_ballot_w64(cm != 0) != 0;
    pend_rbase = rbase;
  }
  if (pend_any)
    for (int ql = 0; ql < QPW; ++ql) {
      if (ql < nq_w) process_query(ql, lists[0]);
      rotate();
    }
#pragma unroll
  for (int ql = 0; ql < QPW; ++ql) {
    if (ql >= nq_w) continue;
    const int64_t q = q0 + 4 * ql + wave;
    float* ds = part_s + (q * n_parts + p) * (int64_t)k;
    int64_t* di = part_i + (q * n_parts + p) * (int64_t)k;
#pragma unroll
    for (int j = 0; j < NS; ++j) {
      const int pos = 64 * j + lane;
      if (pos < k) {
        const int idx = lists[ql].i[j];
        ds[pos] = lists[ql].s[j];
        di[pos] = idx >= 0 ? index_base + r_begin + idx : -1;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// GEMM plan (many queries: the scan is bound by the matrix cores)
// ---------------------------------------------------------------------------
// The store is taken in chunks of rows.  For each chunk the 256 x 256 block
// GEMM core computes the fp32 score matrix S[q][r] into the workspace (sized
// to stay in the MALL), then one workgroup per query selects that chunk's
// top k exactly:
//  * a strided sample of RS_SMP scores is sorted; the sample at a rank
//    chosen so that ~2k + 256 scores are expected above it is a threshold tau;
//  * one pass collects the scores >= tau into LDS (counting them all); if
//    there are at least k of them the top k are all among them (the k-th
//    best is >= tau), and if at most RS_CAP a bitonic sort orders them by
//    (score desc, index asc) and the first k are the chunk's list;
//  * otherwise tau moves by bisection over the sample ranks (more passes);
//    if no rank works (a chunk of massive ties or one ordered against the
//    sample), k arg-max passes over the chunk give the same list exactly.
// Chunks of at most 4096 rows are sorted whole.  NaN and -inf scores are
// never selected; lists are padded with (-inf, -1).  Chunk lists are merged
// by the common merge kernel.
constexpr int RS_CAP = 2048;  // candidates sorted per (query, chunk)
constexpr int RS_SMP = 1024;  // threshold samples
constexpr int RS_SEG = 64;    // chunk rows per score segment (one maximum each)
constexpr int64_t RS_MAXCHUNK = 262144;  // rows of the largest chunk (its segment tables sit in LDS)
constexpr int RS_MAXSEG = (int)(RS_MAXCHUNK / RS_SEG);  // segments of the largest chunk

// v of another lane of the same row of 16 (DPP control C, full masks)
template <int C>
__device__ inline float dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), C, 0xf, 0xf, false));
}

// Epilogue of a score tile.  A wave's columns are 64-row segments of the
// chunk (accumulator column blocks 4 g .. 4 g + 3 form segment g); the 16
// lanes that share a query row reduce each segment's maximum, which is
// stored for the selection.  With a bound from earlier chunks (running k-th
// best score of the query), a segment whose maximum is below it cannot
// contribute and is not written.  bound(row) gives the bound of the tile's
// query row.
template <typename Core, typename Bound>
__device__ inline void score_tile_store(const Core& core, int64_t q0, int64_t nq, int64_t c0,
                                        int64_t nr, float* __restrict__ S, int64_t lds,
                                        float* __restrict__ segmax, int64_t n_seg, Bound bound) {
  constexpr int NJ = Core::NJ, NG = NJ / 4;
  const int lane = threadIdx.x & 63;
  const int64_t seg0 = c0 / RS_SEG + Core::col_base() / RS_SEG;
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = Core::row_of(i, r);
      float m[NG];
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        float v = -__builtin_inff();
#pragma unroll
        for (int jj = 0; jj < 4; ++jj)
          if (Core::col_of(4 * g + jj) < nr) v = fmaxf(v, core.acc[i][4 * g + jj][r]);
        // rotations within each row of 16 lanes (DPP row_ror 8, 4, 2, 1)
        v = fmaxf(v, dpp_f<0x128>(v));
        v = fmaxf(v, dpp_f<0x124>(v));
        v = fmaxf(v, dpp_f<0x122>(v));
        v = fmaxf(v, dpp_f<0x121>(v));
        m[g] = v;
      }
      if (row < nq) {
        const float b = bound(row);
        if ((lane & 15) == 0) {
#pragma unroll
          for (int g = 0; g < NG; ++g) segmax[(q0 + row) * n_seg + seg0 + g] = m[g];
        }
        float* dst = S + (q0 + row) * lds + c0;
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          const int col = Core::col_of(j);
          if (col < nr && !(m[j >> 2] < b)) dst[col] = core.acc[i][j][r];
        }
      }
    }
}

// Scores of one chunk of store rows: items are (query tile, row tile) pairs.
// XCD x (workgroup b goes to XCD b % 8) takes a contiguous range of items,
// query tile fastest: the query tiles of one row tile read the same store
// rows through the same L2.  NT (a single query tile): every store row is
// read once, with the non-temporal cache policy.
template <typename Tag, bool NT>
__global__ __launch_bounds__(256) void score_gemm_kernel(
    const _Float16* __restrict__ Q, int64_t n_q, int64_t ldq, const _Float16* __restrict__ G,
    int64_t nc, int64_t ldg, int n_qt, int n_items, int per_xcd, int n_st,
    float* __restrict__ S, int64_t lds, float* __restrict__ segmax, int64_t n_seg,
    const float* __restrict__ thr, int use_bound) {
  __shared__ GemmSmem sm;
  const int item = (int)(blockIdx.x & 7u) * per_xcd + (int)(blockIdx.x >> 3);
  if (item >= n_items) return;  // uniform
  const int qt = item % n_qt, rt = item / n_qt;
  const int64_t q0 = (int64_t)qt * GT, c0 = (int64_t)rt * GT;
  int64_t nq = n_q - q0, nr = nc - c0;
  nq = nq > GT ? GT : nq;
  nr = nr > GT ? GT : nr;
  const i32x4 dq = make_desc(Q + q0 * ldq, (uint32_t)(nq * ldq * 2));
  const i32x4 dg = make_desc(G + c0 * ldg, (uint32_t)(nr * ldg * 2));
  // the tile's query bounds, staged in LDS (the main loop's barriers publish them)
  __shared__ float tb[GT];
  tb[threadIdx.x] = use_bound && q0 + threadIdx.x < n_q ? thr[q0 + threadIdx.x] : -__builtin_inff();
  GemmCore<Tag, NT> core;
  core.zero();
  core.run(sm, dq, ldq, dg, ldg, n_st);
  score_tile_store(core, q0, nq, c0, nr, S, lds, segmax, n_seg, [&](int row) { return tb[row]; });
}

// The same with 128-query x 256-row tiles on the three-slot ring
// (GemmCoreR): for query counts whose last 256-query tile would be at most
// half used.
template <typename Tag, bool NT>
__global__ __launch_bounds__(256) void score_gemm_r_kernel(
    const _Float16* __restrict__ Q, int64_t n_q, int64_t ldq, const _Float16* __restrict__ G,
    int64_t nc, int64_t ldg, int n_qt, int n_items, int per_xcd, int n_st,
    float* __restrict__ S, int64_t lds, float* __restrict__ segmax, int64_t n_seg,
    const float* __restrict__ thr, int use_bound) {
  __shared__ GemmSmemR sm;
  const int item = (int)(blockIdx.x & 7u) * per_xcd + (int)(blockIdx.x >> 3);
  if (item >= n_items) return;  // uniform
  const int qt = item % n_qt, rt = item / n_qt;
  const int64_t q0 = (int64_t)qt * GRQ, c0 = (int64_t)rt * GRR;
  int64_t nq = n_q - q0, nr = nc - c0;
  nq = nq > GRQ ? GRQ : nq;
  nr = nr > GRR ? GRR : nr;
  // this wave's 64 store rows
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  int64_t nw = nr - 64 * wave;
  nw = nw < 0 ? 0 : (nw > 64 ? 64 : nw);
  const i32x4 dq = make_desc(Q + q0 * ldq, (uint32_t)(nq * ldq * 2));
  const i32x4 dg = make_desc(G + (c0 + 64 * wave) * ldg, (uint32_t)(nw * ldg * 2));
  // the tile's query bounds, staged in LDS (the ring's barriers publish them)
  __shared__ float tb[GRQ];
  if (threadIdx.x < GRQ)
    tb[threadIdx.x] = use_bound && q0 + threadIdx.x < n_q ? thr[q0 + threadIdx.x] : -__builtin_inff();
  GemmCoreR<Tag, NT> core;
  core.zero();
  core.run(sm, dq, ldq, dg, ldg, n_st);
  score_tile_store(core, q0, nq, c0, nr, S, lds, segmax, n_seg, [&](int row) { return tb[row]; });
}

// Order-preserving key of a float (larger float, larger key).  Selectable
// scores are those above -inf and not NaN: keys in (fkey(-inf), fkey(+inf)].
__device__ inline uint32_t fkey(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ inline float fkey_inv(uint32_t key) {
  return __uint_as_float((key & 0x80000000u) ? (key & 0x7fffffffu) : ~key);
}
__device__ inline bool selectable(uint32_t key) { return key > 0x007fffffu && key <= 0xff800000u; }
// (score desc, index asc) as one descending 64-bit key; 0 is padding
__device__ inline uint64_t rs_key(uint32_t key, int64_t j) {
  return ((uint64_t)key << 32) | (uint64_t)(0xffffffffu - (uint32_t)j);
}

// Descending bitonic sort of n (a power of two) keys in LDS, 256 threads.
template <typename T>
__device__ inline void bitonic_desc(T* a, int n) {
  for (int size = 2; size <= n; size <<= 1)
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      __syncthreads();
      for (int t = threadIdx.x; t < n / 2; t += 256) {
        const int i = 2 * t - (t & (stride - 1));
        const int j = i + stride;
        const T x = a[i], y = a[j];
        const bool down = (i & size) == 0;
        if (down ? (x < y) : (x > y)) {
          a[i] = y;
          a[j] = x;
        }
      }
    }
  __syncthreads();
}

__device__ inline uint64_t block_max_u64(uint64_t v, uint64_t* red) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)v, off, kWave);
    const uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(v >> 32), off, kWave);
    const uint64_t o = ((uint64_t)hi << 32) | lo;
    v = o > v ? o : v;
  }
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  uint64_t m = red[0];
#pragma unroll
  for (int w = 1; w < 4; ++w) m = red[w] > m ? red[w] : m;
  return m;
}

__global__ __launch_bounds__(256) void score_rselect_kernel(
    const float* __restrict__ S, int64_t lds, const float* __restrict__ segmax, int64_t n_seg,
    float* __restrict__ thr, int64_t nc, int k, int part, int n_parts, int64_t index_base,
    float* __restrict__ part_s, int64_t* __restrict__ part_i) {
  __shared__ uint64_t cand[RS_CAP];
  __shared__ uint32_t smp[RS_MAXSEG];  // segment maxima or samples, sorted
  __shared__ uint16_t segs[RS_MAXSEG];
  __shared__ uint64_t red_u[4];
  __shared__ int n_cand, n_pass;
  const int64_t q = blockIdx.x;
  const int t = threadIdx.x;
  const float* s = S + q * lds;
  const float* sm = segmax + q * n_seg;
  const int n_sc = (int)((nc + RS_SEG - 1) / RS_SEG);
  float* ds = part_s + (q * n_parts + part) * (int64_t)k;
  int64_t* di = part_i + (q * n_parts + part) * (int64_t)k;

  // Bound from this call's earlier chunks, all of lower index: the running
  // maximum of their k-th scores has k entries at or above it that precede
  // every row of this chunk, so only scores strictly above it can still
  // enter the top k.  Segments whose maximum is below it were not written.
  const float bnd = part > 0 ? thr[q] : -__builtin_inff();
  const uint32_t bkey = fkey(bnd);
  const bool has_b = part > 0 && selectable(bkey);
  const uint32_t floor_key = has_b ? bkey + 1u : 0x00800000u;
  const float floor_f = fkey_inv(floor_key);  // NaN when the bound is +inf: nothing passes

  // collect every selectable score >= tau (up to RS_CAP of them), reading
  // only the segments whose maximum reaches tau; returns how many there are
  auto take = [&](float v, int64_t j, uint32_t tau) {
    const uint32_t key = fkey(v);
    if (selectable(key) && key >= tau) {
      const int p = atomicAdd(&n_cand, 1);
      if (p < RS_CAP) cand[p] = rs_key(key, j);
    }
  };
  auto collect = [&](uint32_t tau) -> int {
    const float tau_f = fkey_inv(tau);  // the float whose key is tau
    __syncthreads();
    if (t == 0) {
      n_cand = 0;
      n_pass = 0;
    }
    __syncthreads();
    for (int g = t; g < n_sc; g += 256)
      if (sm[g] >= tau_f) segs[atomicAdd(&n_pass, 1)] = (uint16_t)g;
    __syncthreads();
    const int np = n_pass;
    // 16 threads per segment (16 bytes each), SB segments per group in flight
    constexpr int SB = 4;
    const int grp = t >> 4, l16 = t & 15;
    const f32x4* s4 = reinterpret_cast<const f32x4*>(s);  // rows are 1 KB aligned
    for (int e0 = 0; e0 < np; e0 += 16 * SB) {
      f32x4 v[SB];
      int64_t j0[SB];
#pragma unroll
      for (int u = 0; u < SB; ++u) {
        const int e = e0 + 16 * u + grp;
        j0[u] = e < np ? (int64_t)segs[e] * RS_SEG + 4 * l16 : -1;
        // a segment's 64 columns lie inside the row (lds is a multiple of 256)
        v[u] = j0[u] >= 0 ? s4[j0[u] >> 2]
                          : f32x4{-__builtin_inff(), -__builtin_inff(), -__builtin_inff(),
                                  -__builtin_inff()};
      }
#pragma unroll
      for (int u = 0; u < SB; ++u) {
        const float m = fmaxf(fmaxf(v[u][0], v[u][1]), fmaxf(v[u][2], v[u][3]));
        if (j0[u] >= 0 && m >= tau_f) {
#pragma unroll
          for (int e4 = 0; e4 < 4; ++e4)
            if (j0[u] + e4 < nc) take(v[u][e4], j0[u] + e4, tau);
        }
      }
    }
    __syncthreads();
    return n_cand;
  };

  bool ok = false;
  int c = 0;
  if (nc <= RS_CAP || has_b) {
    c = collect(floor_key);  // everything above the bound
    ok = c <= RS_CAP;        // fewer than k entries is allowed
  } else {
    // No bound yet: the k-th largest segment maximum.  k segments reach it,
    // so at least k scores do; unless one segment holds many of the top
    // scores, few more than k do.
    int n_sort = 64;
    while (n_sort < n_sc) n_sort <<= 1;
    for (int g = t; g < n_sort; g += 256) {
      const uint32_t key = g < n_sc ? fkey(sm[g]) : 0u;
      smp[g] = selectable(key) ? key : 0u;
    }
    bitonic_desc(smp, n_sort);
    const uint32_t tau = k <= n_sc && smp[k - 1] ? smp[k - 1] : floor_key;
    c = collect(tau);
    ok = c <= RS_CAP;
  }
  if (!ok) {
    {
      uint32_t v[RS_SMP / 256];
#pragma unroll
      for (int u = 0; u < RS_SMP / 256; ++u) {
        const int64_t j = (int64_t)(u * 256 + t) * nc / RS_SMP;
        const bool written = !has_b || sm[j / RS_SEG] >= floor_f;
        const uint32_t key = written ? fkey(s[j]) : 0u;
        v[u] = selectable(key) && key >= floor_key ? key : 0u;
      }
#pragma unroll
      for (int u = 0; u < RS_SMP / 256; ++u) smp[u * 256 + t] = v[u];
    }
    bitonic_desc(smp, RS_SMP);
    int lo = 0, hi = RS_SMP - 1;
    int rho = (int)(((int64_t)(2 * k + 256) * RS_SMP + nc - 1) / nc) - 1;
    rho = rho < 0 ? 0 : (rho > hi ? hi : rho);
    while (lo <= hi) {
      const uint32_t tau = smp[rho];
      if (tau == 0u) {  // fewer selectable samples than rho + 1
        hi = rho - 1;
      } else {
        c = collect(tau);
        if (c >= k && c <= RS_CAP) {
          ok = true;
          break;
        }
        if (c < k) lo = rho + 1;
        else hi = rho - 1;
      }
      rho = (lo + hi) / 2;
    }
  }
  float kth = -__builtin_inff();
  if (ok) {
    int n_sort = 64;  // power of two >= max(c, k)
    while (n_sort < c || n_sort < k) n_sort <<= 1;
    for (int j = c + t; j < n_sort; j += 256) cand[j] = 0ull;
    bitonic_desc(cand, n_sort);
    for (int j = t; j < k; j += 256) {
      const uint64_t e = cand[j];
      ds[j] = e ? fkey_inv((uint32_t)(e >> 32)) : -__builtin_inff();
      di[j] = e ? index_base + (int64_t)(0xffffffffu - (uint32_t)e) : -1;
    }
    const uint64_t e = cand[k - 1];
    kth = e ? fkey_inv((uint32_t)(e >> 32)) : -__builtin_inff();
  } else {
    // exact: the r-th entry is the largest key (above the floor) below the
    // (r-1)-th
    uint64_t prev = ~0ull;
    for (int r = 0; r < k; ++r) {
      uint64_t best = 0ull;
      if (prev != 0ull)
        for (int64_t j = t; j < nc; j += 256) {
          if (has_b && !(sm[j / RS_SEG] >= floor_f)) continue;  // not written
          const uint32_t key = fkey(s[j]);
          if (selectable(key) && key >= floor_key) {
            const uint64_t e = rs_key(key, j);
            if (e < prev && e > best) best = e;
          }
        }
      best = block_max_u64(best, red_u);
      if (t == 0) {
        ds[r] = best ? fkey_inv((uint32_t)(best >> 32)) : -__builtin_inff();
        di[r] = best ? index_base + (int64_t)(0xffffffffu - (uint32_t)best) : -1;
      }
      if (r == k - 1 && best) kth = fkey_inv((uint32_t)(best >> 32));
      prev = best;
    }
  }
  // running bound for the next chunk (its GEMM skips segments below it)
  if (t == 0) thr[q] = has_b && bnd > kth ? bnd : kth;
}

// ---------------------------------------------------------------------------
// split-K plan
// ---------------------------------------------------------------------------
// Partial scores of (query block, row tile, D-slice) -> spart[slice][q][row]
// (nqp = 64 n_qb query rows of n_g scores per slice).
template <bool F16>
__global__ __launch_bounds__(256) void score_splitk_kernel(
    const char* __restrict__ Q, int64_t n_q, int64_t ldq, const char* __restrict__ G,
    int64_t n_g, int64_t ldg, int n_grp, int n_qb, int n_tiles, int n_split,
    float* __restrict__ spart) {
  const int64_t nqp = (int64_t)n_qb * SQB;
  constexpr int EB = STag<F16>::bytes;
  __shared__ i32x4 xpose[4][2 * 128];
  uint32_t b = blockIdx.x;
  const int qb = (int)(b % (uint32_t)n_qb);
  b /= (uint32_t)n_qb;
  const int tile = (int)(b % (uint32_t)n_tiles);
  const int split = (int)(b / (uint32_t)n_tiles);
  const int g_begin = (int)((int64_t)n_grp * split / n_split);
  const int g_end = (int)((int64_t)n_grp * (split + 1) / n_split);
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int lane = threadIdx.x & 63;
  const int64_t q0 = (int64_t)qb * SQB;
  int64_t nq_blk = n_q - q0;
  nq_blk = nq_blk > SQB ? SQB : nq_blk;
  const __amdgpu_buffer_rsrc_t rq = make_rsrc(Q + q0 * ldq * EB, (uint32_t)(nq_blk * ldq * EB));
  const int64_t r0 = (int64_t)tile * STN + 32 * wave;
  int64_t nrow = n_g - r0;
  nrow = nrow < 0 ? 0 : (nrow > 32 ? 32 : nrow);
  const __amdgpu_buffer_rsrc_t rg = make_rsrc(G + r0 * ldg * EB, (uint32_t)(nrow * ldg * EB));
  f32x4 acc[4][2];
#pragma unroll
  for (int qt = 0; qt < 4; ++qt)
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) acc[qt][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
  score_tile<F16>(rq, ldq, rg, ldg, g_begin, g_end, lane, &xpose[wave][0], acc);
  float* dst = spart + (int64_t)split * n_g * nqp;
#pragma unroll
  for (int qt = 0; qt < 4; ++qt)
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t q = q0 + 16 * qt + 4 * (lane >> 4) + r;
        const int64_t row = r0 + 16 * rt + (lane & 15);
        if (row < n_g) dst[q * n_g + row] = acc[qt][rt][r];
      }
}

// ---------------------------------------------------------------------------
// merge
// ---------------------------------------------------------------------------
struct Cand {
  float s;
  int64_t i;
};

__device__ inline Cand cand_none() { return Cand{-__builtin_inff(), -1}; }

__device__ inline bool better(const Cand& a, const Cand& b) {
  if (a.i < 0) return false;
  if (b.i < 0) return true;
  return a.s > b.s || (a.s == b.s && a.i < b.i);
}

__device__ inline Cand wave_best(Cand c) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    Cand o;
    o.s = __shfl_xor(c.s, off, kWave);
    o.i = __shfl_xor(c.i, off, kWave);
    if (better(o, c)) c = o;
  }
  return c;
}

// One workgroup per query: k rounds of block arg-max over the source heads.
// Split-K plan with at most 256 store rows (a batch of new rows scored and
// merged into a running list): one wave per query sums the slices of its
// scores in slice order and takes the k best of those rows and of the
// previous list (merge) by k rounds of wave arg-max, writing the list in
// place.  Replaces the partition select and the merge launches.
__global__ __launch_bounds__(64) void score_small_select_kernel(
    const float* __restrict__ spart, int64_t nqp, int64_t n_g, int n_split, int k, int merge,
    int64_t index_base, float* top_s, int64_t* top_i) {
  const int64_t q = blockIdx.x;
  const int lane = threadIdx.x;
  const int64_t plane = n_g * nqp;
  Cand c[6];
  // rows lane + 64 m; slices summed in order, 8 slices of all four rows in
  // flight at once
  float acc[4];
  bool live[4];
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    live[m] = lane + 64 * m < n_g;
    acc[m] = live[m] ? spart[q * n_g + lane + 64 * m] : 0.f;
  }
  int sp = 1;
  for (; sp + 8 <= n_split; sp += 8) {
    float x[4][8];
#pragma unroll
    for (int m = 0; m < 4; ++m)
#pragma unroll
      for (int u = 0; u < 8; ++u)
        x[m][u] = live[m] ? spart[(sp + u) * plane + q * n_g + lane + 64 * m] : 0.f;
#pragma unroll
    for (int m = 0; m < 4; ++m)
#pragma unroll
      for (int u = 0; u < 8; ++u) acc[m] += x[m][u];
  }
  for (; sp < n_split; ++sp)
#pragma unroll
    for (int m = 0; m < 4; ++m)
      if (live[m]) acc[m] += spart[sp * plane + q * n_g + lane + 64 * m];
#pragma unroll
  for (int m = 0; m < 4; ++m)  // NaN and -inf are never selected
    c[m] = live[m] && acc[m] > -__builtin_inff() ? Cand{acc[m], index_base + lane + 64 * m}
                                                 : Cand{-__builtin_inff(), -1};
#pragma unroll
  for (int m = 0; m < 2; ++m) {
    const int e = lane + 64 * m;
    c[4 + m] = Cand{-__builtin_inff(), -1};
    if (merge && e < k) c[4 + m] = Cand{top_s[q * k + e], top_i[q * k + e]};
  }
  for (int r = 0; r < k; ++r) {
    Cand lb = c[0];
#pragma unroll
    for (int m = 1; m < 6; ++m)
      if (better(c[m], lb)) lb = c[m];
    const Cand wb = wave_best(lb);
    if (lane == 0) {
      top_s[q * k + r] = wb.i >= 0 ? wb.s : -__builtin_inff();
      top_i[q * k + r] = wb.i;
    }
    if (wb.i >= 0) {
#pragma unroll
      for (int m = 0; m < 6; ++m)
        if (c[m].i == wb.i && c[m].s == wb.s) c[m].i = -1;  // indices are unique
    }
  }
}

// Up to 4 sources per thread: n_parts + merge <= 1024.
constexpr int MERGE_SPT = 4;
constexpr int MERGE_CAP = 2048;  // entries gathered and sorted in LDS
constexpr int MERGE_ROUNDS_K = 24;  // k up to this: k arg-max rounds are faster than the sorts

// Bitonic sort of n (a power of two, <= MERGE_CAP) candidates, best first
// ((score desc, index asc), empty entries last).
__device__ inline void bitonic_cand(Cand* a, int n) {
  for (int size = 2; size <= n; size <<= 1)
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      __syncthreads();
      for (int t = threadIdx.x; t < n / 2; t += 256) {
        const int i = 2 * t - (t & (stride - 1));
        const int j = i + stride;
        const Cand x = a[i], y = a[j];
        if ((i & size) == 0 ? better(y, x) : better(x, y)) {
          a[i] = y;
          a[j] = x;
        }
      }
    }
  __syncthreads();
}

// Split-K plan with more than 256 rows (a store of fewer than 32768 rows):
// one workgroup per (query, part of at most 8192 rows).  Pass 1 sums every
// row's slices (slice order, 32 loads in flight per thread) into LDS and
// keeps the best row of each 16-row segment; tau, the k-th best of those
// maxima, is reached by k distinct rows, so the k best of the part are at
// or above it (with fewer than k segments every row qualifies).  Pass 2
// gathers the rows at or above tau, and the previous list when merging
// into a single part, into LDS; a bitonic sort orders them and the first k
// are the part's list (random stores: ~1-2 k rows): the answer itself for a
// single part, else a partition list for the merge kernel.  Should more
// than SPL_CAP rows qualify (massive ties) the list is built by k rounds of
// block arg-max instead.
constexpr int SPL_SEG = 16;
constexpr int SPL_CAP = MERGE_CAP - 128;  // gathered rows (the previous list takes <= 128 more)
constexpr int SPL_PART = 8192;            // rows per part: their scores stay in LDS
constexpr int SPL_SLD = 8;                // slices loaded at once

__global__ __launch_bounds__(256) void score_split_topk_kernel(
    const float* __restrict__ spart, int64_t nqp, int64_t n_g, int n_split, int k, int merge,
    int64_t index_base, int n_parts, float* __restrict__ part_s, int64_t* __restrict__ part_i,
    float* top_s, int64_t* top_i) {
  __shared__ Cand buf[MERGE_CAP];  // segment maxima, then candidates, then (fallback) the list
  __shared__ float sc[SPL_PART];
  __shared__ Cand wbest[4];
  __shared__ int cnt;
  const int64_t q = blockIdx.x / (uint32_t)n_parts;
  const int p = (int)(blockIdx.x % (uint32_t)n_parts);
  const int t = threadIdx.x;
  const int64_t r0 = (int64_t)p * SPL_PART;
  int64_t nr = n_g - r0;
  nr = nr > SPL_PART ? SPL_PART : nr;
  const int64_t plane = n_g * nqp;
  const float* base = spart + q * n_g + r0;
  const int64_t ib = index_base + r0;
  const bool direct = n_parts == 1;  // the part's list is the answer
  const bool with_prev = direct && merge;
  // the scores of rows j0 + 256 u (u < 4), slices summed in order per row
  auto scores4 = [&](int64_t j0) -> f32x4 {
    f32x4 v = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int sp = 0; sp < n_split; sp += SPL_SLD) {
      f32x4 x[SPL_SLD];
#pragma unroll
      for (int a = 0; a < SPL_SLD; ++a)
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int64_t j = j0 + 256 * u;
          x[a][u] = j < nr && sp + a < n_split ? base[(sp + a) * plane + j] : 0.f;
        }
#pragma unroll
      for (int a = 0; a < SPL_SLD; ++a) v += x[a];
    }
    return v;
  };
  // NaN and -inf are never selected
  auto cand_of = [&](float v, int64_t j) -> Cand {
    return j < nr && v > -__builtin_inff() ? Cand{v, ib + j} : cand_none();
  };
  const int n_seg = (int)((nr + SPL_SEG - 1) / SPL_SEG);  // <= SPL_PART / SPL_SEG
  for (int64_t jb = 0; jb < nr; jb += 1024) {
    const f32x4 v = scores4(jb + t);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t j = jb + 256 * u + t;
      if (j < nr) sc[j] = v[u];
      Cand c = cand_of(v[u], j);
#pragma unroll
      for (int off = 8; off >= 1; off >>= 1) {
        Cand o;
        o.s = __shfl_xor(c.s, off, kWave);
        o.i = __shfl_xor(c.i, off, kWave);
        if (better(o, c)) c = o;
      }
      const int seg = (int)((jb + 256 * u) / SPL_SEG) + t / SPL_SEG;
      if ((t & (SPL_SEG - 1)) == 0 && seg < n_seg) buf[seg] = c;
    }
  }
  int n1 = 1;
  while (n1 < n_seg) n1 <<= 1;
  for (int e = n_seg + t; e < n1; e += 256) buf[e] = cand_none();
  bitonic_cand(buf, n1);
  const Cand tau = k <= n_seg ? buf[k - 1] : cand_none();
  __syncthreads();
  if (t == 0) cnt = 0;
  __syncthreads();
  for (int64_t j = t; j < nr; j += 256) {
    const Cand c = cand_of(sc[j], j);
    if (c.i >= 0 && !better(tau, c)) {
      const int pos = atomicAdd(&cnt, 1);
      if (pos < SPL_CAP) buf[pos] = c;
    }
  }
  __syncthreads();
  int n = cnt;
  float* os = direct ? top_s + q * k : part_s + (q * n_parts + p) * (int64_t)k;
  int64_t* oi = direct ? top_i + q * k : part_i + (q * n_parts + p) * (int64_t)k;
  if (n <= SPL_CAP) {
    if (with_prev) {
      for (int e = t; e < k; e += 256) {
        const Cand c{top_s[q * k + e], top_i[q * k + e]};
        buf[n + e] = c.i >= 0 ? c : cand_none();
      }
      n += k;
    }
    int n2 = 1;
    while (n2 < n || n2 < k) n2 <<= 1;
    for (int e = n + t; e < n2; e += 256) buf[e] = cand_none();
    bitonic_cand(buf, n2);
    for (int j = t; j < k; j += 256) {
      const Cand c = buf[j];
      os[j] = c.i >= 0 ? c.s : -__builtin_inff();
      oi[j] = c.i >= 0 ? c.i : -1;
    }
    return;
  }
  // fallback: round r takes the best candidate strictly after round r - 1's
  Cand last = cand_none();
  for (int r = 0; r < k; ++r) {
    Cand tb = cand_none();
    for (int64_t j = t; j < nr; j += 256) {
      const Cand c = cand_of(sc[j], j);
      if (c.i >= 0 && (r == 0 || better(last, c)) && better(c, tb)) tb = c;
    }
    if (with_prev)
      for (int e = t; e < k; e += 256) {
        const Cand c{top_s[q * k + e], top_i[q * k + e]};
        if (c.i >= 0 && (r == 0 || better(last, c)) && better(c, tb)) tb = c;
      }
    const Cand wb = wave_best(tb);
    if ((t & 63) == 0) wbest[t >> 6] = wb;
    __syncthreads();
    Cand best = wbest[0];
#pragma unroll
    for (int w = 1; w < 4; ++w)
      if (better(wbest[w], best)) best = wbest[w];
    if (t == 0) buf[r] = best;
    last = best;
    __syncthreads();
  }
  for (int j = t; j < k; j += 256) {
    const Cand c = buf[j];
    os[j] = c.i >= 0 ? c.s : -__builtin_inff();
    oi[j] = c.i >= 0 ? c.i : -1;
  }
}

// One workgroup per query.  Every source list is sorted, so with d =
// ceil(k / sources) the first d entries of all sources hold at least k
// entries, and the k-th best of them, tau, is a lower bound on the k-th
// best overall.  The entries at or above tau (a prefix of each source) are
// gathered into LDS and sorted; the first k are the merged list (random
// sources: ~k to 2k entries).  For small k, and past MERGE_CAP such entries
// (massive ties), the merge is k rounds of block arg-max over the source
// heads instead (at k = 100 over 512 sources: ~37 us against ~150 us; at
// k = 10 the rounds take ~13 us against ~15-25 us).
__global__ __launch_bounds__(256) void score_merge_kernel(const float* __restrict__ part_s,
                                                          const int64_t* __restrict__ part_i,
                                                          int n_parts, int k, int merge,
                                                          float* top_s, int64_t* top_i) {
  __shared__ Cand wb[4];
  __shared__ float os[256];
  __shared__ int64_t oi[256];
  __shared__ Cand buf[MERGE_CAP];
  __shared__ int cnt;
  const int64_t q = blockIdx.x;
  const int t = threadIdx.x;
  const int n_src = n_parts + (merge ? 1 : 0);
  const float* src_s[MERGE_SPT];
  const int64_t* src_i[MERGE_SPT];
  int head[MERGE_SPT];
  Cand cur[MERGE_SPT];
#pragma unroll
  for (int m = 0; m < MERGE_SPT; ++m) {
    const int src = t + 256 * m;
    src_s[m] = nullptr;
    src_i[m] = nullptr;
    if (src < n_parts) {
      src_s[m] = part_s + (q * n_parts + src) * (int64_t)k;
      src_i[m] = part_i + (q * n_parts + src) * (int64_t)k;
    } else if (src < n_src) {
      src_s[m] = top_s + q * (int64_t)k;
      src_i[m] = top_i + q * (int64_t)k;
    }
    head[m] = 0;
    cur[m] = src_s[m] ? Cand{src_s[m][0], src_i[m][0]} : Cand{-__builtin_inff(), -1};
  }
  const Cand none{-__builtin_inff(), -1};
  if (k > MERGE_ROUNDS_K) {
    // tau: the k-th best of the first d entries of every source
    const int d = n_src > 0 ? (k + n_src - 1) / n_src : 1;
    int n1 = 1;
    while (n1 < n_src * d) n1 <<= 1;
    for (int e = t; e < n1; e += 256) {
      const int src = e / d, j = e - src * d;
      Cand c = none;
      if (src < n_src) {
        const float* ps = src < n_parts ? part_s + (q * n_parts + src) * (int64_t)k : top_s + q * (int64_t)k;
        const int64_t* pi = src < n_parts ? part_i + (q * n_parts + src) * (int64_t)k : top_i + q * (int64_t)k;
        c = Cand{ps[j], pi[j]};
      }
      buf[e] = c;
    }
    bitonic_cand(buf, n1);
    const Cand tau = buf[k - 1];
    if (t == 0) cnt = 0;
    __syncthreads();
    // gather the entries at or above tau (every valid one when tau is empty),
    // four entries of a source per load round
#pragma unroll
    for (int m = 0; m < MERGE_SPT; ++m) {
      if (!src_s[m]) continue;
      bool go = true;
      for (int j0 = 0; go && j0 < k; j0 += 4) {
        Cand e4[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) e4[u] = j0 + u < k ? Cand{src_s[m][j0 + u], src_i[m][j0 + u]} : none;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          if (!go) break;
          if (e4[u].i < 0 || better(tau, e4[u])) {
            go = false;
          } else {
            const int pos = atomicAdd(&cnt, 1);
            if (pos < MERGE_CAP) buf[pos] = e4[u];
          }
        }
      }
    }
    __syncthreads();
    const int n = cnt;
    if (n <= MERGE_CAP) {
      int n2 = 1;
      while (n2 < n || n2 < k) n2 <<= 1;
      for (int e = n + t; e < n2; e += 256) buf[e] = none;
      bitonic_cand(buf, n2);
      for (int j = t; j < k; j += 256) {
        const Cand c = buf[j];
        top_s[q * (int64_t)k + j] = c.i >= 0 ? c.s : -__builtin_inff();
        top_i[q * (int64_t)k + j] = c.i >= 0 ? c.i : -1;
      }
      return;
    }
  }
  for (int j = 0; j < k; ++j) {
    // this thread's best head
    Cand tb = cur[0];
    int tm = 0;
#pragma unroll
    for (int m = 1; m < MERGE_SPT; ++m)
      if (better(cur[m], tb)) {
        tb = cur[m];
        tm = m;
      }
    Cand b = wave_best(tb);
    if ((t & 63) == 0) wb[t >> 6] = b;
    __syncthreads();
    Cand best = wb[0];
#pragma unroll
    for (int w = 1; w < 4; ++w)
      if (better(wb[w], best)) best = wb[w];
    if (t == 0) {
      os[j] = best.i >= 0 ? best.s : -__builtin_inff();
      oi[j] = best.i;
    }
    // the source whose head won advances (indices are unique across sources)
    if (best.i >= 0 && tb.i == best.i && tb.s == best.s) {
#pragma unroll
      for (int m = 0; m < MERGE_SPT; ++m)
        if (m == tm) {
          ++head[m];
          cur[m] = head[m] < k ? Cand{src_s[m][head[m]], src_i[m][head[m]]} : Cand{-__builtin_inff(), -1};
        }
    }
    __syncthreads();
  }
  for (int j = t; j < k; j += 256) {
    top_s[q * (int64_t)k + j] = os[j];
    top_i[q * (int64_t)k + j] = oi[j];
  }
}

}  // namespace

// Streaming-plan launch shape: list capacity KMAX (64 or 128: one or two
// list registers per query), ring depth RING, K-groups per stage GPS, list
// slots per wave QPW (a block's queries / 4: register budget), workgroups
// per CU and tile height TR x 64 rows.  The lists live in registers, so the
// LDS holds only the ring (RING x GPS x (64 TR + 64) rows x 128 B); two
// workgroups per CU were 10-20% faster than one at k > 64, and 128-row
// tiles (a three-stage ring of 24 KB slots) beat 64-row tiles (four 16 KB
// slots) by 4% at 16 queries and 13% at 64 (2M x 8192 fp16: 78-83% of HBM
// bandwidth at 16 to 64 queries and k up to 128).
struct StreamCfg {
  int kmax, ring, gps, qpw, per_cu, tr;
};
static StreamCfg stream_cfg(int64_t n_q, int k) {
  const int64_t qb = n_q < SQ ? n_q : SQ;
  const int qpw = qb <= 16 ? 4 : (qb <= 32 ? 8 : 16);
  const int kmax = k <= 64 ? 64 : 128;
  // 128-row tiles: half the query bytes per store byte through the ring
  return {kmax, 3, 1, qpw, 2, 2};
}

static size_t align256(size_t b) { return (b + 255) / 256 * 256; }
constexpr int64_t BOUND_ROWS = 16384;  // prefix rows whose segment maxima bound the k-th best

ScorePlan plan_score(int64_t n_q, int64_t n_g, int64_t D, int k, int elem_bytes) {
  ScorePlan P{};
  P.D = D;
  P.n_qb = (int)((n_q + SQB - 1) / SQB);
  P.n_grp = (int)(D * elem_bytes / 128);
  if (n_q <= 0 || n_g <= 0) return P;
  // (the streaming plan at 128-384 queries measured 1.2-2.8x slower)
  // GEMM plan: score chunks of at most ~256 MB (MALL-resident between the
  // GEMM and the selection) and RS_MAXCHUNK rows, at most GEMM_MAX_PARTS
  // chunks (the merge takes 1024 sources, one of them the previous list);
  // a store too large for that takes the streaming plan, whose partitions
  // grow with the store
  constexpr int64_t GEMM_MAX_PARTS = 1023;
  if (elem_bytes == 2 && D % GKS == 0 && n_q >= 128 && n_g >= 4096 &&
      n_g <= RS_MAXCHUNK * GEMM_MAX_PARTS) {
    // Tiles: 256 x 256, or 128 queries x 256 rows (the ring core) where the
    // last 256-query tile would be at most half used (n_q % 256 in [1, 128])
    // and the query count is small enough that store rows, not queries, set
    // the work (the narrow tile reads each store row once per 128 queries).
    const int64_t rem = n_q % 256;
    const bool narrow = rem >= 1 && rem <= 128 && n_q <= 384;
    const int64_t rt = narrow ? GRR : GT;
    int64_t chunk = ((int64_t)256 << 20) / (n_q * 4);
    chunk = chunk > RS_MAXCHUNK ? RS_MAXCHUNK : chunk;
    const int64_t min_chunk = (n_g + GEMM_MAX_PARTS - 1) / GEMM_MAX_PARTS;  // <= RS_MAXCHUNK
    chunk = chunk < min_chunk ? min_chunk : chunk;
    chunk = chunk < 4096 ? 4096 : chunk;
    chunk = (chunk + rt - 1) / rt * rt;
    const int64_t all = (n_g + rt - 1) / rt * rt;
    chunk = chunk > all ? all : chunk;
    P.gemm = narrow ? 2 : 1;
    P.chunk = chunk;
    P.n_parts = (int)((n_g + chunk - 1) / chunk);
    P.rows_per_part = chunk;
    P.split = 1;
    // scores, segment maxima (one per 64 rows), running bound per query
    P.spart_bytes = (size_t)n_q * (size_t)chunk * 4 + (size_t)n_q * (size_t)(chunk / RS_SEG) * 4 +
                    (size_t)n_q * 4;
    P.list_entries = (size_t)n_q * (size_t)P.n_parts * (size_t)k;
    return P;
  }
  const int64_t n_tiles = (n_g + STN - 1) / STN;
  // Too few (query block, row tile) pairs to occupy 256 CUs: split D.
  int64_t split = 1;
  if (P.n_qb * n_tiles < 256) {
    split = (256 + P.n_qb * n_tiles - 1) / (P.n_qb * n_tiles);
    const int64_t max_split = P.n_grp / 8 > 1 ? P.n_grp / 8 : 1;  // >= 8 groups per slice
    split = split > max_split ? max_split : split;
    const int64_t cap = ((int64_t)256 << 20) / ((int64_t)n_g * P.n_qb * SQB * 4);
    split = split > cap ? cap : split;
  }
  if (split >= 2) {
    // partial slices, then one selection workgroup per query straight into
    // the output (no partition lists): n_g < 256 x 128 rows here
    P.split = (int)split;
    P.n_tiles = (int)n_tiles;
    P.rows_per_part = SPL_PART;
    P.n_parts = (int)((n_g + SPL_PART - 1) / SPL_PART);
    if (P.n_parts == 1) P.n_parts = 0;  // one part: its list is the answer (no partition lists)
    P.spart_bytes = (size_t)split * (size_t)n_g * (size_t)P.n_qb * SQB * 4;
  } else {
    P.split = 1;
    // streaming plan: 64 queries per workgroup; two workgroups per CU when
    // the ring and the lists fit in half the LDS, else one; as many
    // partitions as workgroups fit at once (an exact multiple of the CU
    // count: 248 workgroups ran ~13% slower than 256 on k <= 32)
    P.n_qb = (int)((n_q + SQ - 1) / SQ);
    int64_t per_wave = (int64_t)stream_cfg(n_q, k).per_cu * 256;
    per_wave = per_wave > 1016 ? 1016 : per_wave;  // the merge takes <= 1024 sources
    int64_t parts = (per_wave + P.n_qb - 1) / P.n_qb;
    const int64_t srt = (int64_t)SR * stream_cfg(n_q, k).tr;  // rows per tile
    const int64_t t64 = (n_g + srt - 1) / srt;
    parts = parts > t64 ? t64 : parts;
    parts = parts > per_wave ? per_wave : (parts < 1 ? 1 : parts);
    int64_t rpp = (n_g + parts - 1) / parts;
    rpp = (rpp + srt - 1) / srt * srt;
    P.rows_per_part = rpp;
    P.n_parts = (int)((n_g + rpp - 1) / rpp);
    P.spart_bytes = 0;
    // the bound pass (~0.1 ms) pays when the lists see many insertions: a
    // large store and many (query, list entry) pairs
    if (n_g >= 16 * BOUND_ROWS && n_q * k >= 1024) {
      P.bound_rows = BOUND_ROWS;
      const size_t nb = (size_t)(BOUND_ROWS / SR);
      P.spart_bytes = align256((size_t)n_q * nb * 4) + align256((size_t)n_q * nb * 8) + align256((size_t)n_q * 4);
    }
  }
  P.list_entries = (size_t)n_q * (size_t)P.n_parts * (size_t)k;
  return P;
}

// bound[q] = k-th largest of the nb segment maxima of query q (-inf when
// fewer than k are finite).  One workgroup per query; nb <= 1024.
__global__ __launch_bounds__(256) void score_bound_kernel(const float* __restrict__ seg_s, int nb, int k,
                                                          float* __restrict__ bound) {
  __shared__ float v[1024];
  const int64_t q = blockIdx.x;
  for (int i = threadIdx.x; i < 1024; i += 256) v[i] = i < nb ? seg_s[q * nb + i] : -__builtin_inff();
  __syncthreads();
  bitonic_desc(v, 1024);
  if (threadIdx.x == 0) bound[q] = v[k - 1];
}

hipError_t launch_score_topk(bool f16, const ScorePlan& plan, const void* Q, int64_t n_q,
                             int64_t ldq, const void* G, int64_t n_g, int64_t ldg, int k,
                             int64_t index_base, int merge, float* top_s, int64_t* top_i,
                             float* part_s, int64_t* part_i, float* spart, hipStream_t s) {
  const int n_parts = n_g > 0 ? plan.n_parts : 0;
  if (n_g > 0 && plan.gemm) {
    const int tq = plan.gemm == 2 ? GRQ : GT, tr = plan.gemm == 2 ? GRR : GT;
    const int n_qt = (int)((n_q + tq - 1) / tq);
    const int n_st = plan.n_grp;  // 64-element fp16 stages (128 bytes)
    const int64_t n_seg = plan.chunk / RS_SEG;
    float* segmax = spart + n_q * plan.chunk;
    float* thr = segmax + n_q * n_seg;
    for (int c = 0; c < plan.n_parts; ++c) {
      const int64_t r0 = (int64_t)c * plan.chunk;
      const int64_t nc = n_g - r0 < plan.chunk ? n_g - r0 : plan.chunk;
      const int n_items = n_qt * (int)((nc + tr - 1) / tr);
      const int per_xcd = (n_items + 7) / 8;
      const bool nt = n_qt == 1;
      hipLaunchKernelGGL(plan.gemm == 2 ? (nt ? score_gemm_r_kernel<F16Tag, true>
                                              : score_gemm_r_kernel<F16Tag, false>)
                                        : (nt ? score_gemm_kernel<F16Tag, true>
                                              : score_gemm_kernel<F16Tag, false>),
                         dim3((unsigned)(8 * per_xcd)), dim3(256), 0, s, (const _Float16*)Q, n_q,
                         ldq, (const _Float16*)G + r0 * ldg, nc, ldg, n_qt, n_items, per_xcd, n_st,
                         spart, plan.chunk, segmax, n_seg, (const float*)thr, c > 0 ? 1 : 0);
      hipLaunchKernelGGL(score_rselect_kernel, dim3((unsigned)n_q), dim3(256), 0, s,
                         (const float*)spart, plan.chunk, (const float*)segmax, n_seg, thr, nc, k, c,
                         plan.n_parts, index_base + r0, part_s, part_i);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  } else if (n_g > 0 && plan.split <= 1) {
    // lower bound on each query's k-th best score: the k-th largest of the
    // maxima of the first bound_rows / 64 row segments (k distinct rows reach
    // it).  The maxima come from this kernel run with k = 1 over one-tile
    // partitions.
    const float* bound = nullptr;
    if (plan.bound_rows > 0) {
      const int nb = (int)(plan.bound_rows / SR);
      char* w = reinterpret_cast<char*>(spart);
      float* seg_s = reinterpret_cast<float*>(w);
      int64_t* seg_i = reinterpret_cast<int64_t*>(w + align256((size_t)n_q * nb * 4));
      float* bnd = reinterpret_cast<float*>(w + align256((size_t)n_q * nb * 4) + align256((size_t)n_q * nb * 8));
      const StreamCfg cb = stream_cfg(n_q, 1);
      const int pp = (nb + 7) / 8 * 8;
      dim3 gb((unsigned)(plan.n_qb * pp)), bb(256);
      bool ok = false;
#define ATTR_SB(KM, RG, GP, QW)                                                                  \
  if (cb.qpw == QW) {                                                                          \
    ok = true;                                                                                   \
    if (f16)                                                                                     \
      hipLaunchKernelGGL((score_stream_kernel<true, KM, RG, GP, QW, 1>), gb, bb, 0, s,           \
                         (const char*)Q, n_q, ldq, (const char*)G, plan.bound_rows, ldg,        \
                         plan.n_grp, 1, (int64_t)SR, nb, plan.n_qb, (const float*)nullptr, seg_s, \
                         seg_i, (int64_t)0);                                                     \
    else                                                                                         \
      hipLaunchKernelGGL((score_stream_kernel<false, KM, RG, GP, QW, 1>), gb, bb, 0, s,          \
                         (const char*)Q, n_q, ldq, (const char*)G, plan.bound_rows, ldg,        \
                         plan.n_grp, 1, (int64_t)SR, nb, plan.n_qb, (const float*)nullptr, seg_s, \
                         seg_i, (int64_t)0);                                                     \
  }
      ATTR_SB(64, 4, 1, 4)
      ATTR_SB(64, 4, 1, 8)
      ATTR_SB(64, 4, 1, 16)
#undef ATTR_SB
      if (!ok) return hipErrorInvalidConfiguration;
      hipLaunchKernelGGL(score_bound_kernel, dim3((unsigned)n_q), dim3(256), 0, s, (const float*)seg_s, nb,
                         k, bnd);
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
      bound = bnd;
    }
    const int parts_pad = (plan.n_parts + 7) / 8 * 8;
    dim3 grid((unsigned)(plan.n_qb * parts_pad)), block(256);
#define ATTR_SS(KM, RG, GP, QW, TRR)                                                             \
  if (c.kmax == KM && c.ring == RG && c.gps == GP && c.qpw == QW && c.tr == TRR) {               \
    launched = true;                                                                             \
    if (f16)                                                                                     \
      hipLaunchKernelGGL((score_stream_kernel<true, KM, RG, GP, QW, TRR>), grid, block, 0, s,     \
                         (const char*)Q, n_q, ldq, (const char*)G, n_g, ldg, plan.n_grp, k,      \
                         plan.rows_per_part, plan.n_parts, plan.n_qb, bound, part_s, part_i,     \
                         index_base);                                                            \
    else                                                                                         \
      hipLaunchKernelGGL((score_stream_kernel<false, KM, RG, GP, QW, TRR>), grid, block, 0, s,    \
                         (const char*)Q, n_q, ldq, (const char*)G, n_g, ldg, plan.n_grp, k,      \
                         plan.rows_per_part, plan.n_parts, plan.n_qb, bound, part_s, part_i,     \
                         index_base);                                                            \
  }
    const StreamCfg c = stream_cfg(n_q, k);
    bool launched = false;
    ATTR_SS(64, 3, 1, 4, 2)
    ATTR_SS(64, 3, 1, 8, 2)
    ATTR_SS(64, 3, 1, 16, 2)
    ATTR_SS(128, 3, 1, 4, 2)
    ATTR_SS(128, 3, 1, 8, 2)
    ATTR_SS(128, 3, 1, 16, 2)
    if (!launched) return hipErrorInvalidConfiguration;
#undef ATTR_SS
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  } else if (n_g > 0) {
    dim3 grid((unsigned)((int64_t)plan.n_qb * plan.n_tiles * plan.split)), block(256);
    if (f16)
      hipLaunchKernelGGL(score_splitk_kernel<true>, grid, block, 0, s, (const char*)Q, n_q, ldq,
                         (const char*)G, n_g, ldg, plan.n_grp, plan.n_qb, plan.n_tiles, plan.split,
                         spart);
    else
      hipLaunchKernelGGL(score_splitk_kernel<false>, grid, block, 0, s, (const char*)Q, n_q, ldq,
                         (const char*)G, n_g, ldg, plan.n_grp, plan.n_qb, plan.n_tiles, plan.split,
                         spart);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (n_g <= 256) {
      hipLaunchKernelGGL(score_small_select_kernel, dim3((unsigned)n_q), dim3(64), 0, s,
                         (const float*)spart, (int64_t)plan.n_qb * SQB, n_g, plan.split, k,
                         merge, index_base, top_s, top_i);
      return hipGetLastError();
    }
    const int np = plan.n_parts > 0 ? plan.n_parts : 1;
    hipLaunchKernelGGL(score_split_topk_kernel, dim3((unsigned)(n_q * np)), dim3(256), 0, s,
                       (const float*)spart, (int64_t)plan.n_qb * SQB, n_g, plan.split, k, merge,
                       index_base, np, part_s, part_i, top_s, top_i);
    e = hipGetLastError();
    if (e != hipSuccess || np == 1) return e;
  }
  hipLaunchKernelGGL(score_merge_kernel, dim3((unsigned)n_q), dim3(256), 0, s,
                     (const float*)part_s, (const int64_t*)part_i, n_parts, k, merge, top_s, top_i);
  return hipGetLastError();
}

}  // namespace attr
