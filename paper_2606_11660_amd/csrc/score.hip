// Query x gradient-store scoring with exact streaming top-k (section
// "Attribution Pipelines": every gradient store supports exact top-k lookup
// of the most influential items).
//
// score_partial: a workgroup owns QB = 64 queries and one contiguous
// partition of store rows, walked in tiles of 128 rows.  The 64 x 128 score
// tile is a matrix-core GEMM over D (fp16 16x16x32 or fp32 16x16x4 MFMA,
// fp32 accumulate); store rows are streamed with line-coalesced loads and
// transposed through LDS into MFMA fragments (as in the projection), query
// fragments come from L2.  The tile goes to LDS and one lane per query
// walks it in row order against the query's running threshold, inserting
// winners into a sorted per-query list in LDS.  Rows are visited in
// increasing index order, so a strict ">" keeps the lower index on ties.
// The Q x N score matrix is never written to memory.
//
// score_merge: one workgroup per query merges the sorted partition lists
// (and the previous result when merging a new store chunk) by repeated
// block-wide arg-max, ordering by (score desc, index asc).
#include "common.h"
#include "kernels.h"

namespace attr {
namespace {

constexpr int SQB = 64;    // queries per workgroup
constexpr int STN = 128;   // store rows per tile (4 waves x 32 rows)
constexpr int SPD = 3;     // 128-byte K-groups of store loads in flight
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

template <bool F16, int KMAX>
__global__ __launch_bounds__(256) void score_partial_kernel(
    const char* __restrict__ Q, int64_t n_q, int64_t ldq, const char* __restrict__ G,
    int64_t n_g, int64_t ldg, int64_t D, int k, int64_t rows_per_part, int n_parts,
    int n_qb, float* __restrict__ part_s, int64_t* __restrict__ part_i, int64_t index_base) {
  using Tag = typename STag<F16>::tag;
  constexpr int EB = STag<F16>::bytes;
  constexpr int E = 16 / EB;
  constexpr int KS = 4 * E;
  constexpr int KG = 2 * KS;  // elements per 128-byte group

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
  // merge-lane state (wave 0, lane = query)
  int cnt = 0;
  float thr = -__builtin_inff();
  __syncthreads();

  int64_t nq_blk = n_q - q0;
  nq_blk = nq_blk > SQB ? SQB : nq_blk;
  const __amdgpu_buffer_rsrc_t rq = make_rsrc(Q + q0 * ldq * EB, (uint32_t)(nq_blk * ldq * EB));

  // store-row load mapping (line-coalesced) and LDS transpose slots
  const int lrow = lane >> 3, lch = lane & 7;
  const uint32_t g_base = (uint32_t)((int64_t)lrow * ldg * EB + lch * 16);
  const uint32_t g_half = (uint32_t)(8 * ldg * EB);
  const uint32_t g_tile = (uint32_t)(16 * ldg * EB);
  const int wslot = lrow * 8 + (lch ^ lrow);
  const int ri = lane & 15, rgrp = lane >> 4;
  const int rslot0 = ri * 8 + (rgrp ^ (ri & 7));
  const int rslot1 = ri * 8 + ((4 + rgrp) ^ (ri & 7));
  // query fragment offsets
  const uint32_t q_base = (uint32_t)(((int64_t)ri * ldq + E * rgrp) * EB);
  const uint32_t q_tile = (uint32_t)(16 * ldq * EB);
  i32x4* xp = &xpose[wave][0];
  const int n_grp = (int)(D / KG);

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
      if (u < n_grp) issue_g(u, gbuf[u]);
    issue_q(0, qcur);

    for (int g0 = 0; g0 < n_grp; g0 += SPD) {
#pragma unroll
      for (int u = 0; u < SPD; ++u) {
        const int grp = g0 + u;
        if (grp + SPD - 1 < n_grp) issue_g(grp + SPD - 1, gbuf[(u + SPD - 1) % SPD]);
        if (grp < n_grp) {
          if (grp + 1 < n_grp) issue_q(grp + 1, qnxt);
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

    // scores -> LDS: lane holds query 16 qt + 4 (lane / 16) + r, row 16 rt + lane % 16
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
      const int q = lane;
      for (int j = 0; j < (int)nvalid; ++j) {
        const float s = sc[q][j];
        if (s > thr) {
          int pos = cnt < k ? cnt : k - 1;
          while (pos > 0 && ls[q][pos - 1] < s) {
            ls[q][pos] = ls[q][pos - 1];
            li[q][pos] = li[q][pos - 1];
            --pos;
          }
          ls[q][pos] = s;
          li[q][pos] = (int)(r0 + j);
          if (cnt < k) ++cnt;
          if (cnt == k) thr = ls[q][k - 1];
        }
      }
    }
    __syncthreads();
  }

  if (wave == 0 && lane < nq_blk) {
    const int64_t q = q0 + lane;
    float* ds = part_s + (q * n_parts + p) * (int64_t)k;
    int64_t* di = part_i + (q * n_parts + p) * (int64_t)k;
    for (int j = 0; j < k; ++j) {
      ds[j] = ls[lane][j];
      di[j] = li[lane][j] >= 0 ? index_base + li[lane][j] : -1;
    }
  }
}

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

int score_parts(int64_t n_q, int64_t n_g) {
  const int64_t n_qb = (n_q + SQB - 1) / SQB;
  int64_t parts = (512 + n_qb - 1) / n_qb;
  const int64_t max_parts = (n_g + STN - 1) / STN;
  if (parts > max_parts) parts = max_parts;
  if (parts > 255) parts = 255;
  if (parts < 1) parts = 1;
  return (int)parts;
}

int64_t score_rows_per_part(int64_t n_g, int parts) {
  int64_t rpp = (n_g + parts - 1) / parts;
  return (rpp + STN - 1) / STN * STN;
}

hipError_t launch_score_topk(bool f16, const void* Q, int64_t n_q, int64_t ldq, const void* G,
                             int64_t n_g, int64_t ldg, int64_t D, int k, int64_t index_base,
                             int merge, float* top_s, int64_t* top_i, float* part_s,
                             int64_t* part_i, hipStream_t s) {
  int n_parts = 0;
  if (n_g > 0) {
    n_parts = score_parts(n_q, n_g);
    const int64_t rpp = score_rows_per_part(n_g, n_parts);
    n_parts = (int)((n_g + rpp - 1) / rpp);
    const int n_qb = (int)((n_q + SQB - 1) / SQB);
    dim3 grid((unsigned)(n_qb * n_parts)), block(256);
#define ATTR_SP(F, KM)                                                                         \
  hipLaunchKernelGGL((score_partial_kernel<F, KM>), grid, block, 0, s, (const char*)Q, n_q, ldq, \
                     (const char*)G, n_g, ldg, D, k, rpp, n_parts, n_qb, part_s, part_i,        \
                     index_base)
    if (f16) {
      if (k <= 16) ATTR_SP(true, 16);
      else ATTR_SP(true, 128);
    } else {
      if (k <= 16) ATTR_SP(false, 16);
      else ATTR_SP(false, 128);
    }
#undef ATTR_SP
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(score_merge_kernel, dim3((unsigned)n_q), dim3(256), 0, s,
                     (const float*)part_s, (const int64_t*)part_i, n_parts, k, merge, top_s, top_i);
  return hipGetLastError();
}

}  // namespace attr
