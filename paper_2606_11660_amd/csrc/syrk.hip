// Full second-moment accumulation H += X^T X over store rows (the flat
// autocorrelation / empirical Fisher preconditioner of the method-family
// table; TrackStar's Fisher fitting step in section "Attribution Pipelines").
//
// The contraction runs over rows of X (K = row index), so the operands are
// K-major: the GEMM core for K-major operands reads 64-row x 256-column
// stages of X itself and transposes them while reading its MFMA fragments
// out of LDS (no transposed copy of X is written).  Only the upper-triangle
// tiles (tp <= tq) of X^T X are computed.  Rows are taken in equal chunks
// of at most 524288; a chunk is split into 16 K-slices computed by separate
// workgroups (at D = 8192, 528 tiles x 16 slices are 33 whole rounds of the
// 256 CUs; chunks of 65536 rows left a quarter-full last round and took 5%
// longer), and only the slices that hold rows are launched.  Slice results
// go to fp32 partial tiles and a reduce kernel adds them, in slice order,
// into an fp64 accumulator (at 10^6 x 8192 the reduce of two chunks costs
// ~1 ms, of four 1.9 ms); the last chunk's reduce rounds its sums straight
// into H.  Precision: fp32 MFMA accumulation over at most
// 32768 rows, fp64 across slices and chunks, one rounding into H at the end
// of the call (the spectrum of H spans ~6 decades on low-rank-plus-noise
// stores, and long fp32 accumulation visibly perturbs its small eigenvalues;
// sampled entries of H at 10^6 x 8192 are within 5e-7 of fp64, relative to
// the largest).
// Deterministic: fixed tile, slice and chunk orders, no atomics.
#include "common.h"
#include "gemm.h"
#include "kernels.h"
#include "syrk_plan.h"

namespace attr {
namespace {

static_assert(kSyrkTile == GT, "the plan's tile is the GEMM core's");
constexpr int TILE_E = GT * GT;  // elements per tile

// Upper-triangle tile u -> (tp, tq), tp <= tq, row-major over tp.
__device__ inline void upper_tile(int u, int nt, int& tp, int& tq) {
  int p = 0;
  while (u >= nt - p) {
    u -= nt - p;
    ++p;
  }
  tp = p;
  tq = p + u;
}

// Upper-triangle tile v in band order: bands of 4 tile rows, each walked
// column by column (the rows of a band first), so that consecutive tiles
// share their row blocks.
__device__ inline void band_tile(int v, int nt, int& tp, int& tq) {
  tp = 0;
  tq = 0;
  for (int b0 = 0; b0 < nt; b0 += 4) {
    const int bh = nt - b0 < 4 ? nt - b0 : 4;
    const int cnt = bh * (bh + 1) / 2 + (nt - b0 - bh) * bh;
    if (v < cnt) {
      for (int q = b0; q < nt; ++q) {
        const int c = q - b0 + 1 < bh ? q - b0 + 1 : bh;
        if (v < c) {
          tp = b0 + v;
          tq = q;
          return;
        }
        v -= c;
      }
    }
    v -= cnt;
  }
}

// Work item of workgroup b: workgroups go to the 8 XCDs round robin
// (b % 8).  The K-slices are taken one after the other by the whole chip
// (even slices first, then odd), so that the rows being read at any time
// are one slice's (512 MB at 8192 columns); within a slice XCD x takes the
// contiguous band-ordered tile range [x per_xcd, (x + 1) per_xcd), so the
// workgroups resident on one XCD share row blocks through its L2.
template <typename Tag, typename T>
__global__ __launch_bounds__(256) void syrk_kernel(const T* __restrict__ X, int64_t ldx,
                                                   int64_t n_rows, int64_t r0, int64_t D, int nt,
                                                   int n_up, int J, int per_xcd, int64_t Cs,
                                                   float* __restrict__ part) {
  __shared__ GemmSmem sm;
  const int l = (int)(blockIdx.x >> 3);
  // slices in the order 0, 2, 4, ..., then 1, 3, 5, ...: the even (plain) and
  // odd (negated, slower) slices meet only once per launch, instead of at
  // every slice boundary, where workgroups of both kinds share an XCD and
  // drift apart (which broke the L2 sharing of row blocks: 63.5 -> 91.8 GB
  // of L2-miss traffic per 500000-row launch with the slices in plain order)
  const int o = l / per_xcd;
  const int ne = (J + 1) >> 1;  // even slices
  const int j = o < ne ? 2 * o : 2 * (o - ne) + 1;
  const int v = (int)(blockIdx.x & 7u) * per_xcd + (l - o * per_xcd);
  if (o >= J || v >= n_up) return;  // uniform
  int tp, tq;
  band_tile(v, nt, tp, tq);
  const int u = tp * nt - tp * (tp - 1) / 2 + (tq - tp);  // row-major upper index
  // slice j: rows [rs, rs + nr) of X; operand rows start at the tile's
  // first column.  The descriptor range ends at the slice's last row (or at
  // the matrix end, column D of row n_rows - 1): K-rows past it read zeros;
  // columns past D of a row read the next row's values, which only reach
  // outputs of columns >= D (never stored).
  const int64_t rs = r0 + (int64_t)j * Cs;
  int64_t nr = n_rows - rs;
  nr = nr > Cs ? Cs : nr;
  auto range = [&](int64_t c0) -> uint32_t {
    if (nr <= 0) return 0u;
    const int64_t lim_slice = nr * ldx, lim_mat = (n_rows - 1 - rs) * ldx + (D - c0);
    return (uint32_t)((lim_slice < lim_mat ? lim_slice : lim_mat) * 2);
  };
  const int64_t ca = (int64_t)tp * GT, cb = (int64_t)tq * GT;
  const i32x4 da = make_desc(X + rs * ldx + ca, range(ca));
  const i32x4 db = make_desc(X + rs * ldx + cb, range(cb));
  // odd slices accumulate -X^T X (B fragments negated) and store the negated
  // sum: the matrix core's accumulation rounds toward -infinity on average,
  // so the odd slices' sums come out high by about as much as the even
  // slices' come out low, and the fp64 sum over slices cancels the bias
  const int n_st = (int)((nr + GKS - 1) / GKS);  // stages holding rows
  float* dst = part + ((int64_t)j * n_up + u) * TILE_E;
  auto store = [&](const f32x4 (&acc)[8][8], float sgn) {
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int jj = 0; jj < 8; ++jj)
#pragma unroll
        for (int r = 0; r < 4; ++r) dst[((i * 8 + jj) * 4 + r) * 256 + threadIdx.x] = sgn * acc[i][jj][r];
  };
  if (j & 1) {
    GemmCoreT<Tag, true> core;
    core.zero();
    core.run(sm, da, db, ldx, n_st);
    store(core.acc, -1.f);
  } else {
    GemmCoreT<Tag, false> core;
    core.zero();
    core.run(sm, da, db, ldx, n_st);
    store(core.acc, 1.f);
  }
}

// h64[u][e] += sum_j part[j][u][e], slices in order (fragment-order layout).
// Four elements per thread: the J partial vectors (read once, non-temporal)
// are all in flight before the sums are formed.
__global__ __launch_bounds__(256) void syrk_reduce_kernel(const float* __restrict__ part, int J,
                                                          int64_t n_e, double* __restrict__ h64) {
  const int64_t e4 = (int64_t)blockIdx.x * 256 + threadIdx.x;  // n_e is a multiple of 4
  if (4 * e4 >= n_e) return;
  const f32x4* p4 = reinterpret_cast<const f32x4*>(part);
  const int64_t n4 = n_e / 4;
  double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0;
  int j = 0;
  for (; j + 8 <= J; j += 8) {
    f32x4 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = __builtin_nontemporal_load(p4 + (int64_t)(j + u) * n4 + e4);
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      s0 += (double)v[u].x;
      s1 += (double)v[u].y;
      s2 += (double)v[u].z;
      s3 += (double)v[u].w;
    }
  }
  for (; j < J; ++j) {
    const f32x4 v = __builtin_nontemporal_load(p4 + (int64_t)j * n4 + e4);
    s0 += (double)v.x;
    s1 += (double)v.y;
    s2 += (double)v.z;
    s3 += (double)v.w;
  }
  double* h = h64 + 4 * e4;
  h[0] += s0;
  h[1] += s1;
  h[2] += s2;
  h[3] += s3;
}

__global__ __launch_bounds__(256) void fill_zero_kernel(double* __restrict__ p, int64_t n) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e < n) p[e] = 0.0;
}

// The last chunk's reduce and the store in one pass: for element f of tile u,
// s = sum_j part[j][u][f] (fp64, slices in order, as syrk_reduce_kernel), t =
// h64[u][f] + s when earlier chunks left sums in h64 (else t = s), then
// H[p][q] = fp32(H[p][q] + t) for p <= q: one rounding into H, with the same
// operations in the same order as a separate reduce into h64 followed by a
// store, but without h64's fill, write and re-read on single-chunk calls.
// Fragment-order element f of tile u maps to (i, jj, r, thread) with row
// 128 (w/2) + 16 i + 4 (lane/16) + r and column 128 (w%2) + 16 jj + lane%16;
// four consecutive elements per thread share the row, columns adjacent.
__global__ __launch_bounds__(256) void syrk_reduce_store_kernel(const float* __restrict__ part, int J,
                                                                int64_t n_e,
                                                                const double* __restrict__ h64,
                                                                int nt, int64_t D,
                                                                float* __restrict__ H) {
  const int u = blockIdx.y;
  const int64_t f0 = 4 * ((int64_t)blockIdx.x * 256 + threadIdx.x);  // 0 .. TILE_E
  const int64_t e4 = ((int64_t)u * TILE_E + f0) / 4;
  const f32x4* p4 = reinterpret_cast<const f32x4*>(part);
  const int64_t n4 = n_e / 4;
  double s[4] = {0.0, 0.0, 0.0, 0.0};
  int j = 0;
  for (; j + 8 <= J; j += 8) {
    f32x4 v[8];
#pragma unroll
    for (int w = 0; w < 8; ++w) v[w] = __builtin_nontemporal_load(p4 + (int64_t)(j + w) * n4 + e4);
#pragma unroll
    for (int w = 0; w < 8; ++w) {
      s[0] += (double)v[w].x;
      s[1] += (double)v[w].y;
      s[2] += (double)v[w].z;
      s[3] += (double)v[w].w;
    }
  }
  for (; j < J; ++j) {
    const f32x4 v = __builtin_nontemporal_load(p4 + (int64_t)j * n4 + e4);
    s[0] += (double)v.x;
    s[1] += (double)v.y;
    s[2] += (double)v.z;
    s[3] += (double)v.w;
  }
  if (h64) {
    const double* h = h64 + 4 * e4;
#pragma unroll
    for (int c = 0; c < 4; ++c) s[c] = h[c] + s[c];
  }
  int tp, tq;
  upper_tile(u, nt, tp, tq);
  // the thread's four elements share row p and take columns q0 .. q0 + 3
  // (f0 is a multiple of 4): one 16-byte access where all four are stored
  {
    const int th = (int)(f0 & 255), w = th >> 6, lane = th & 63;
    const int irj = (int)(f0 >> 8);
    const int r = irj & 3, jj = (irj >> 2) & 7, i = irj >> 5;
    const int64_t p = (int64_t)tp * GT + 128 * (w >> 1) + 16 * i + 4 * (lane >> 4) + r;
    const int64_t q0 = (int64_t)tq * GT + 128 * (w & 1) + 16 * jj + (lane & 15);
    if ((D & 3) == 0 && p < D && q0 + 3 < D && p <= q0) {
      f32x4* hp = reinterpret_cast<f32x4*>(H + p * D + q0);
      f32x4 hv = *hp;
      hv.x = (float)((double)hv.x + s[0]);
      hv.y = (float)((double)hv.y + s[1]);
      hv.z = (float)((double)hv.z + s[2]);
      hv.w = (float)((double)hv.w + s[3]);
      *hp = hv;
      return;
    }
  }
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int64_t f = f0 + c;
    const int th = (int)(f & 255), w = th >> 6, lane = th & 63;
    const int irj = (int)(f >> 8);
    const int r = irj & 3, jj = (irj >> 2) & 7, i = irj >> 5;
    const int64_t p = (int64_t)tp * GT + 128 * (w >> 1) + 16 * i + 4 * (lane >> 4) + r;
    const int64_t q = (int64_t)tq * GT + 128 * (w & 1) + 16 * jj + (lane & 15);
    if (p < D && q < D && p <= q) {
      float* hp = H + p * D + q;
      *hp = (float)((double)*hp + s[c]);
    }
  }
}

}  // namespace

hipError_t launch_syrk(bool bf16, const void* X, int64_t ldx, int64_t n_rows, int64_t D, float* H,
                       const SyrkPlan& P, void* part, void* h64, hipStream_t s) {
  const int64_t n_e = (int64_t)P.n_up * TILE_E;
  // h64 carries fp64 sums between chunks; a single-chunk call never uses it
  const bool multi = n_rows > P.C;
  hipError_t e;
  if (multi) {
    hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)((n_e + 255) / 256)), dim3(256), 0, s,
                       (double*)h64, n_e);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const int per_xcd = (P.n_up + 7) / 8;  // tiles per XCD and slice
  for (int64_t r0 = 0; r0 < n_rows; r0 += P.C) {
    const int64_t rows = n_rows - r0 < P.C ? n_rows - r0 : P.C;
    const int Jc = (int)((rows + P.Cs - 1) / P.Cs);  // slices holding rows
    dim3 gs((unsigned)(8 * per_xcd * Jc));
    if (bf16)
      hipLaunchKernelGGL((syrk_kernel<Bf16Tag, __bf16>), gs, dim3(256), 0, s, (const __bf16*)X, ldx,
                         n_rows, r0, D, P.nt, P.n_up, Jc, per_xcd, P.Cs, (float*)part);
    else
      hipLaunchKernelGGL((syrk_kernel<F16Tag, _Float16>), gs, dim3(256), 0, s, (const _Float16*)X,
                         ldx, n_rows, r0, D, P.nt, P.n_up, Jc, per_xcd, P.Cs, (float*)part);
    if (r0 + P.C < n_rows)
      hipLaunchKernelGGL(syrk_reduce_kernel, dim3((unsigned)((n_e / 4 + 255) / 256)), dim3(256), 0, s,
                         (const float*)part, Jc, n_e, (double*)h64);
    else
      hipLaunchKernelGGL(syrk_reduce_store_kernel, dim3(TILE_E / 1024, (unsigned)P.n_up), dim3(256),
                         0, s, (const float*)part, Jc, n_e, multi ? (const double*)h64 : nullptr,
                         P.nt, D, H);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace attr
