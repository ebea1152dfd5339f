// Query x gradient-store scoring with exact streaming top-k (section
// "Attribution Pipelines": every gradient store supports exact top-k lookup
// of the most influential items).
//
// Score tiles are 64 queries x 128 store rows, a matrix-core GEMM over D
// (fp16 16x16x32 or fp32 16x16x4 MFMA, fp32 accumulate).  Store rows stream
// with line-coalesced loads and pass through a per-wave LDS tile into MFMA
// fragments (as in the projection); query fragments come from L2.
//
// Two plans, chosen on the host from the problem shape:
//  * fused (large stores): a workgroup owns 64 queries and a contiguous row
//    partition; each finished tile goes to LDS and one lane per query walks
//    it in row order against the query's running threshold, inserting
//    winners into a sorted per-query list in LDS.  Rows are visited in
//    increasing index order, so a strict ">" keeps the lower index on ties.
//    The Q x N score matrix never reaches memory.
//  * split-K (small stores, too few tiles to fill 256 CUs): workgroups own
//    (tile, D-slice) pairs and write fp32 partial scores; a select kernel
//    sums the slices in slice order and runs the same per-query insertion.
// Either way, per-partition sorted lists are merged per query by block-wide
// arg-max in (score desc, index asc) order, which also merges a previous
// result when a store is scored chunk by chunk.
#include "common.h"
#include "kernels.h"

namespace attr {
namespace {

constexpr int SQB = 64;       // queries per workgroup
constexpr int STN = 128;      // store rows per tile (4 waves x 32 rows)
constexpr int SPD = 3;        // 128-byte K-groups of store loads in flight
constexpr int SCP = STN + 4;  // padded score-tile row (bank spread)

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

// Sorted per-query list in LDS, owned by one lane.
template <int KMAX>
struct TopList {
  float (*ls)[KMAX];
  int (*li)[KMAX];
  int cnt;
  float thr;
  __device__ inline void push(int q, int k, float s, int idx) {
    if (!(s > thr)) return;  // NaN never enters; equal scores keep the lower index
    int pos = cnt < k ? cnt : k - 1;
    while (pos > 0 && ls[q][pos - 1] < s) {
      ls[q][pos] = ls[q][pos - 1];
      li[q][pos] = li[q][pos - 1];
      --pos;
    }
    ls[q][pos] = s;
    li[q][pos] = idx;
    if (cnt < k) ++cnt;
    if (cnt == k) thr = ls[q][k - 1];
  }
};

template <int KMAX>
__device__ inline void write_list(float (*ls)[KMAX], int (*li)[KMAX], int q_local, int64_t q,
                                  int p, int n_parts, int k, int64_t index_base,
                                  float* __restrict__ part_s, int64_t* __restrict__ part_i) {
  float* ds = part_s + (q * n_parts + p) * (int64_t)k;
  int64_t* di = part_i + (q * n_parts + p) * (int64_t)k;
  for (int j = 0; j < k; ++j) {
    ds[j] = ls[q_local][j];
    di[j] = li[q_local][j] >= 0 ? index_base + li[q_local][j] : -1;
  }
}

// ---------------------------------------------------------------------------
// fused plan
// ---------------------------------------------------------------------------
template <bool F16, int KMAX>
__global__ __launch_bounds__(256) void score_fused_kernel(
    const char* __restrict__ Q, int64_t n_q, int64_t ldq, const char* __restrict__ G,
    int64_t n_g, int64_t ldg, int n_grp, int k, int64_t rows_per_part, int n_parts, int n_qb,
    float* __restrict__ part_s, int64_t* __restrict__ part_i, int64_t index_base) {
  constexpr int EB = STag<F16>::bytes;
  __shared__ float ls[SQB][KMAX];
  __shared__ int li[SQB][KMAX];
  __shared__ float sc[SQB][SCP];
  __shared__ i32x4 xpose[4][2 * 128];

  const int qb = (int)(blockIdx.x % (uint32_t)n_qb);
  const int p = (int)(blockIdx.x / (uint32_t)n_qb);
  const int64_t q0 = (int64_t)qb * SQB;
  const int64_t r_begin = (int64_t)p * rows_per_part;
  int64_t r_end = r_begin + rows_per_part;
  r_end = r_end > n_g ? n_g : r_end;
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int lane = threadIdx.x & 63;

  for (int e = threadIdx.x; e < SQB * KMAX; e += 256) {
    ls[e / KMAX][e % KMAX] = -__builtin_inff();
    li[e / KMAX][e % KMAX] = -1;
  }
  TopList<KMAX> tl{ls, li, 0, -__builtin_inff()};
  __syncthreads();

  int64_t nq_blk = n_q - q0;
  nq_blk = nq_blk > SQB ? SQB : nq_blk;
  const __amdgpu_buffer_rsrc_t rq = make_rsrc(Q + q0 * ldq * EB, (uint32_t)(nq_blk * ldq * EB));

  for (int64_t r0 = r_begin; r0 < r_end; r0 += STN) {
    int64_t nrow = r_end - (r0 + 32 * wave);
    nrow = nrow < 0 ? 0 : (nrow > 32 ? 32 : nrow);
    const __amdgpu_buffer_rsrc_t rg =
        make_rsrc(G + (r0 + 32 * wave) * ldg * EB, (uint32_t)(nrow * ldg * EB));
    f32x4 acc[4][2];
#pragma unroll
    for (int qt = 0; qt < 4; ++qt)
#pragma unroll
      for (int rt = 0; rt < 2; ++rt) acc[qt][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
    score_tile<F16>(rq, ldq, rg, ldg, 0, n_grp, lane, &xpose[wave][0], acc);
#pragma unroll
    for (int qt = 0; qt < 4; ++qt)
#pragma unroll
      for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          sc[16 * qt + 4 * (lane >> 4) + r][32 * wave + 16 * rt + (lane & 15)] = acc[qt][rt][r];
    __syncthreads();
    if (wave == 0 && lane < nq_blk) {
      int64_t nvalid = r_end - r0;
      nvalid = nvalid > STN ? STN : nvalid;
      for (int j = 0; j < (int)nvalid; ++j) tl.push(lane, k, sc[lane][j], (int)(r0 + j));
    }
    __syncthreads();
  }
  if (wave == 0 && lane < nq_blk)
    write_list<KMAX>(ls, li, lane, q0 + lane, p, n_parts, k, index_base, part_s, part_i);
}

// ---------------------------------------------------------------------------
// split-K plan
// ---------------------------------------------------------------------------
// Partial scores of (query block, row tile, D-slice) -> spart[slice][row][q].
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
        if (row < n_g) dst[row * nqp + q] = acc[qt][rt][r];
      }
}

// One workgroup per (query block, row partition).  For each chunk of 128
// rows the 256 threads sum the slices (slice order, per element) with
// coalesced 16-byte loads into an LDS score tile; then one lane per query
// inserts the chunk in row order.  spart is [slice][row][nqp], nqp = 64 n_qb.
template <int KMAX>
__global__ __launch_bounds__(256) void score_select_kernel(const float* __restrict__ spart,
                                                           int64_t n_q, int64_t nqp, int64_t n_g,
                                                           int n_split, int k,
                                                           int64_t rows_per_part, int n_parts,
                                                           int n_qb, float* __restrict__ part_s,
                                                           int64_t* __restrict__ part_i,
                                                           int64_t index_base) {
  __shared__ float ls[SQB][KMAX];
  __shared__ int li[SQB][KMAX];
  __shared__ float sc[SQB][SCP];
  const int qb = (int)(blockIdx.x % (uint32_t)n_qb);
  const int p = (int)(blockIdx.x / (uint32_t)n_qb);
  const int t = threadIdx.x;
  for (int e = t; e < SQB * KMAX; e += 256) {
    ls[e / KMAX][e % KMAX] = -__builtin_inff();
    li[e / KMAX][e % KMAX] = -1;
  }
  __syncthreads();
  const int64_t q0 = (int64_t)qb * SQB;
  int64_t nq_blk = n_q - q0;
  nq_blk = nq_blk > SQB ? SQB : nq_blk;
  TopList<KMAX> tl{ls, li, 0, -__builtin_inff()};
  const int64_t r0 = (int64_t)p * rows_per_part;
  int64_t r1 = r0 + rows_per_part;
  r1 = r1 > n_g ? n_g : r1;
  const int64_t plane = n_g * nqp;
  const int jr = t >> 1;        // row within the chunk
  const int qh = (t & 1) * 32;  // first of this thread's 32 queries
  for (int64_t c0 = r0; c0 < r1; c0 += STN) {
    int64_t nrow = r1 - c0;
    nrow = nrow > STN ? STN : nrow;
    if (jr < nrow) {
      const f32x4* src = (const f32x4*)(spart + (c0 + jr) * nqp + q0 + qh);
      f32x4 acc[8];
#pragma unroll
      for (int v = 0; v < 8; ++v) acc[v] = src[v];
      int sp = 1;
      for (; sp + 4 <= n_split; sp += 4) {
        f32x4 x[4][8];
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int v = 0; v < 8; ++v) x[u][v] = src[(sp + u) * plane / 4 + v];
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int v = 0; v < 8; ++v) acc[v] += x[u][v];
      }
      for (; sp < n_split; ++sp)
#pragma unroll
        for (int v = 0; v < 8; ++v) acc[v] += src[sp * plane / 4 + v];
#pragma unroll
      for (int v = 0; v < 8; ++v)
#pragma unroll
        for (int e = 0; e < 4; ++e) sc[qh + 4 * v + e][jr] = acc[v][e];
    }
    __syncthreads();
    if (t < nq_blk)
      for (int j = 0; j < (int)nrow; ++j) tl.push(t, k, sc[t][j], (int)(c0 + j));
    __syncthreads();
  }
  if (t < nq_blk) write_list<KMAX>(ls, li, t, q0 + t, p, n_parts, k, index_base, part_s, part_i);
}

// ---------------------------------------------------------------------------
// merge
// ---------------------------------------------------------------------------
struct Cand {
  float s;
  int64_t i;
};

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
__global__ __launch_bounds__(256) void score_merge_kernel(const float* __restrict__ part_s,
                                                          const int64_t* __restrict__ part_i,
                                                          int n_parts, int k, int merge,
                                                          float* top_s, int64_t* top_i) {
  __shared__ Cand wb[4];
  __shared__ float os[256];
  __shared__ int64_t oi[256];
  const int64_t q = blockIdx.x;
  const int t = threadIdx.x;
  const int n_src = n_parts + (merge ? 1 : 0);
  const float* src_s = nullptr;
  const int64_t* src_i = nullptr;
  if (t < n_parts) {
    src_s = part_s + (q * n_parts + t) * (int64_t)k;
    src_i = part_i + (q * n_parts + t) * (int64_t)k;
  } else if (t < n_src) {
    src_s = top_s + q * (int64_t)k;
    src_i = top_i + q * (int64_t)k;
  }
  int head = 0;
  Cand cur{-__builtin_inff(), -1};
  if (src_s) {
    cur.s = src_s[0];
    cur.i = src_i[0];
  }
  for (int j = 0; j < k; ++j) {
    Cand b = wave_best(cur);
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
    if (best.i >= 0 && cur.i == best.i && cur.s == best.s && src_s) {
      ++head;
      if (head < k) {
        cur.s = src_s[head];
        cur.i = src_i[head];
      } else {
        cur.s = -__builtin_inff();
        cur.i = -1;
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

ScorePlan plan_score(int64_t n_q, int64_t n_g, int64_t D, int k, int elem_bytes) {
  ScorePlan P{};
  P.n_qb = (int)((n_q + SQB - 1) / SQB);
  P.n_grp = (int)(D * elem_bytes / 128);
  if (n_q <= 0 || n_g <= 0) return P;
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
    P.split = (int)split;
    P.n_tiles = (int)n_tiles;
    int64_t parts = n_tiles < 255 ? n_tiles : 255;
    int64_t rpp = (n_g + parts - 1) / parts;
    rpp = (rpp + STN - 1) / STN * STN;
    P.rows_per_part = rpp;
    P.n_parts = (int)((n_g + rpp - 1) / rpp);
    P.spart_bytes = (size_t)split * (size_t)n_g * (size_t)P.n_qb * SQB * 4;
  } else {
    P.split = 1;
    int64_t parts = (512 + P.n_qb - 1) / P.n_qb;
    parts = parts > n_tiles ? n_tiles : parts;
    parts = parts > 255 ? 255 : (parts < 1 ? 1 : parts);
    int64_t rpp = (n_g + parts - 1) / parts;
    rpp = (rpp + STN - 1) / STN * STN;
    P.rows_per_part = rpp;
    P.n_parts = (int)((n_g + rpp - 1) / rpp);
    P.spart_bytes = 0;
  }
  P.list_entries = (size_t)n_q * (size_t)P.n_parts * (size_t)k;
  return P;
}

hipError_t launch_score_topk(bool f16, const ScorePlan& plan, const void* Q, int64_t n_q,
                             int64_t ldq, const void* G, int64_t n_g, int64_t ldg, int k,
                             int64_t index_base, int merge, float* top_s, int64_t* top_i,
                             float* part_s, int64_t* part_i, float* spart, hipStream_t s) {
  const int n_parts = n_g > 0 ? plan.n_parts : 0;
  if (n_g > 0 && plan.split <= 1) {
    dim3 grid((unsigned)(plan.n_qb * plan.n_parts)), block(256);
#define ATTR_SF(F, KM)                                                                         \
  hipLaunchKernelGGL((score_fused_kernel<F, KM>), grid, block, 0, s, (const char*)Q, n_q, ldq,   \
                     (const char*)G, n_g, ldg, plan.n_grp, k, plan.rows_per_part, plan.n_parts, \
                     plan.n_qb, part_s, part_i, index_base)
    if (f16) {
      if (k <= 16) ATTR_SF(true, 16);
      else ATTR_SF(true, 128);
    } else {
      if (k <= 16) ATTR_SF(false, 16);
      else ATTR_SF(false, 128);
    }
#undef ATTR_SF
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
    dim3 g2((unsigned)(plan.n_qb * plan.n_parts)), b2(256);
    if (k <= 16)
      hipLaunchKernelGGL(score_select_kernel<16>, g2, b2, 0, s, (const float*)spart, n_q,
                         (int64_t)plan.n_qb * SQB, n_g, plan.split, k, plan.rows_per_part,
                         plan.n_parts, plan.n_qb, part_s, part_i, index_base);
    else
      hipLaunchKernelGGL(score_select_kernel<128>, g2, b2, 0, s, (const float*)spart, n_q,
                         (int64_t)plan.n_qb * SQB, n_g, plan.split, k, plan.rows_per_part,
                         plan.n_parts, plan.n_qb, part_s, part_i, index_base);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(score_merge_kernel, dim3((unsigned)n_q), dim3(256), 0, s,
                     (const float*)part_s, (const int64_t*)part_i, n_parts, k, merge, top_s, top_i);
  return hipGetLastError();
}

}  // namespace attr
