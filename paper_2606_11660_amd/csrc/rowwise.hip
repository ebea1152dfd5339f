// Row-wise processing of compressed gradient rows and the diagonal
// second-moment accumulator.
//
// rowscale: y = unit_normalise(m .* x) cast to the store dtype (the
// "processing" step of section "Attribution Pipelines": unit normalisation
// and the diagonal preconditioner; grad-cosine in the method-family table).
// One workgroup per row; the row stays in registers between the norm and
// the write, so X is read once and Y written once (HBM-bound).
//
// colsumsq: h_j += sum_i x_ij^2, the diagonal of the second moment G^T G.
// Column blocks x row panels; fp32 sums over 8-row groups are added into an
// fp64 accumulator per thread, panel sums are combined in fp64 in panel
// order and rounded once into h (deterministic, no atomics).
#include "common.h"
#include "kernels.h"

namespace attr {
namespace {

template <typename T>
__device__ inline void load8(const T* p, float (&v)[8]);
template <>
__device__ inline void load8<float>(const float* p, float (&v)[8]) {
  const f32x4 a = *(const f32x4*)p;
  const f32x4 b = *(const f32x4*)(p + 4);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
template <>
__device__ inline void load8<_Float16>(const _Float16* p, float (&v)[8]) {
  const f16x8 a = *(const f16x8*)p;
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = (float)a[e];
}
template <>
__device__ inline void load8<__bf16>(const __bf16* p, float (&v)[8]) {
  const bf16x8 a = *(const bf16x8*)p;
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = (float)a[e];
}

// Streaming (non-temporal) load of a row chunk read exactly once.
template <typename T>
__device__ inline void load8_nt(const T* p, float (&v)[8]);
template <>
__device__ inline void load8_nt<float>(const float* p, float (&v)[8]) {
  const f32x4 a = __builtin_nontemporal_load((const f32x4*)p);
  const f32x4 b = __builtin_nontemporal_load((const f32x4*)(p + 4));
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
template <>
__device__ inline void load8_nt<_Float16>(const _Float16* p, float (&v)[8]) {
  const f16x8 a = __builtin_nontemporal_load((const f16x8*)p);
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = (float)a[e];
}
template <>
__device__ inline void load8_nt<__bf16>(const __bf16* p, float (&v)[8]) {
  const i32x4 a = __builtin_nontemporal_load((const i32x4*)p);
  const bf16x8 b = __builtin_bit_cast(bf16x8, a);
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = (float)b[e];
}

template <typename T>
__device__ inline void store8(T* p, const float (&v)[8]);
template <>
__device__ inline void store8<float>(float* p, const float (&v)[8]) {
  __builtin_nontemporal_store(f32x4{v[0], v[1], v[2], v[3]}, (f32x4*)p);
  __builtin_nontemporal_store(f32x4{v[4], v[5], v[6], v[7]}, (f32x4*)(p + 4));
}
template <>
__device__ inline void store8<_Float16>(_Float16* p, const float (&v)[8]) {
  f16x8 a;
#pragma unroll
  for (int e = 0; e < 8; ++e) a[e] = (_Float16)v[e];
  __builtin_nontemporal_store(a, (f16x8*)p);
}

__device__ inline float block_sum256(float v, float* sh) {
  v = wave_sum(v);
  const int wave = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) sh[wave] = v;
  __syncthreads();
  return (sh[0] + sh[1]) + (sh[2] + sh[3]);
}

__device__ inline float row_scale(float ss, int unit) {
  if (!unit) return 1.f;
  return ss > 0.f ? (float)(1.0 / sqrt((double)ss)) : 0.f;
}

// CH > 0: up to CH chunks of 8 elements per thread stay in registers.
// CH == 0: any width, two passes over the row (second pass hits cache).
// seg_e (with row_ss): X holds y 2^-e per 128-column segment, e = seg_e[r * n_ss
// + segment]; the scale of such a segment is 2^e / ||y||.
template <typename TX, typename TY, int CH>
__global__ __launch_bounds__(256) void rowscale_kernel(const TX* __restrict__ X, int64_t ldx,
                                                       int64_t D, const float* __restrict__ m,
                                                       int unit, const float* __restrict__ row_ss,
                                                       const int8_t* __restrict__ seg_e,
                                                       int64_t n_ss, TY* Y, int64_t ldy) {
  __shared__ float sh[4];
  const int64_t r = blockIdx.x;
  const TX* x = X + r * ldx;
  TY* y = Y + r * ldy;
  const int n8 = (int)(D / 8);
  float ss = 0.f;
  if (CH > 0) {
    float v[CH > 0 ? CH : 1][8];
#pragma unroll
    for (int j = 0; j < (CH > 0 ? CH : 1); ++j) {
      const int ch = threadIdx.x + j * 256;
      if (ch < n8) {
        load8_nt<TX>(x + (int64_t)ch * 8, v[j]);
        if (m) {
          float mm[8];
          load8<float>(m + (int64_t)ch * 8, mm);
#pragma unroll
          for (int e = 0; e < 8; ++e) v[j][e] *= mm[e];
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) ss += v[j][e] * v[j][e];
      }
    }
    if (row_ss) {
      ss = 0.f;
      for (int64_t p = 0; p < n_ss; ++p) ss += row_ss[r * n_ss + p];
    } else if (unit) {
      ss = block_sum256(ss, sh);
    }
    const float sc = row_scale(ss, unit);
#pragma unroll
    for (int j = 0; j < (CH > 0 ? CH : 1); ++j) {
      const int ch = threadIdx.x + j * 256;
      if (ch < n8) {
        const float scj = seg_e ? ldexpf(sc, (int)seg_e[r * n_ss + (ch >> 4)]) : sc;
#pragma unroll
        for (int e = 0; e < 8; ++e) v[j][e] *= scj;
        store8<TY>(y + (int64_t)ch * 8, v[j]);
      }
    }
  } else {
    if (row_ss) {
      for (int64_t p = 0; p < n_ss; ++p) ss += row_ss[r * n_ss + p];
    } else if (unit) {
      for (int ch = threadIdx.x; ch < n8; ch += 256) {
        float v[8];
        load8<TX>(x + (int64_t)ch * 8, v);
        if (m) {
          float mm[8];
          load8<float>(m + (int64_t)ch * 8, mm);
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] *= mm[e];
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) ss += v[e] * v[e];
      }
      ss = block_sum256(ss, sh);
    }
    const float sc = row_scale(ss, unit);
    for (int ch = threadIdx.x; ch < n8; ch += 256) {
      float v[8];
      load8<TX>(x + (int64_t)ch * 8, v);
      if (m) {
        float mm[8];
        load8<float>(m + (int64_t)ch * 8, mm);
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] *= mm[e];
      }
      const float scj = seg_e ? ldexpf(sc, (int)seg_e[r * n_ss + (ch >> 4)]) : sc;
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] *= scj;
      store8<TY>(y + (int64_t)ch * 8, v);
    }
  }
}

// Two rows per workgroup (rows 2b and 2b + 1, same column chunks per
// thread): the scale m is read once for both and twice the bytes are in
// flight per workgroup.  Same per-row arithmetic and order as above.
template <typename TX, typename TY, int CH>
__global__ __launch_bounds__(256) void rowscale2_kernel(const TX* __restrict__ X, int64_t ldx,
                                                        int64_t n_rows, int64_t D,
                                                        const float* __restrict__ m, int unit,
                                                        const float* __restrict__ row_ss,
                                                        int64_t n_ss, TY* Y, int64_t ldy) {
  __shared__ float sh[2][4];
  const int64_t r0 = 2 * (int64_t)blockIdx.x;
  const bool two = r0 + 1 < n_rows;
  const int n8 = (int)(D / 8);
  float v[2][CH][8];
  float ss[2] = {0.f, 0.f};
#pragma unroll
  for (int j = 0; j < CH; ++j) {
    const int ch = threadIdx.x + j * 256;
    if (ch < n8) {
      load8_nt<TX>(X + r0 * ldx + (int64_t)ch * 8, v[0][j]);
      if (two) load8_nt<TX>(X + (r0 + 1) * ldx + (int64_t)ch * 8, v[1][j]);
    }
  }
#pragma unroll
  for (int j = 0; j < CH; ++j) {
    const int ch = threadIdx.x + j * 256;
    if (ch < n8) {
      if (m) {
        float mm[8];
        load8<float>(m + (int64_t)ch * 8, mm);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          v[0][j][e] *= mm[e];
          v[1][j][e] *= mm[e];
        }
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        ss[0] += v[0][j][e] * v[0][j][e];
        ss[1] += v[1][j][e] * v[1][j][e];
      }
    }
  }
  if (row_ss) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      ss[h] = 0.f;
      if (h == 0 || two)
        for (int64_t p = 0; p < n_ss; ++p) ss[h] += row_ss[(r0 + h) * n_ss + p];
    }
  } else if (unit) {
    const float a = wave_sum(ss[0]), b = wave_sum(ss[1]);
    if ((threadIdx.x & 63) == 0) {
      sh[0][threadIdx.x >> 6] = a;
      sh[1][threadIdx.x >> 6] = b;
    }
    __syncthreads();
    ss[0] = (sh[0][0] + sh[0][1]) + (sh[0][2] + sh[0][3]);
    ss[1] = (sh[1][0] + sh[1][1]) + (sh[1][2] + sh[1][3]);
  }
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    if (h == 1 && !two) break;
    const float sc = row_scale(ss[h], unit);
    TY* y = Y + (r0 + h) * ldy;
#pragma unroll
    for (int j = 0; j < CH; ++j) {
      const int ch = threadIdx.x + j * 256;
      if (ch < n8) {
#pragma unroll
        for (int e = 0; e < 8; ++e) v[h][j][e] *= sc;
        store8<TY>(y + (int64_t)ch * 8, v[h][j]);
      }
    }
  }
}

template <typename TX, typename TY>
hipError_t launch_rowscale_t(const void* X, int64_t ldx, int64_t n_rows, int64_t D,
                             const float* m, int unit, const float* row_ss, const int8_t* seg_e,
                             int64_t n_ss, void* Y, int64_t ldy, hipStream_t s) {
  dim3 grid((unsigned)n_rows), block(256);
  const int64_t n8 = D / 8;
  const TX* x = (const TX*)X;
  TY* y = (TY*)Y;
#define ATTR_RS(CH) \
  hipLaunchKernelGGL((rowscale_kernel<TX, TY, CH>), grid, block, 0, s, x, ldx, D, m, unit, row_ss, \
                     seg_e, n_ss, y, ldy)
  if (m && !seg_e && n8 <= 1024 && n_rows >= 2) {  // the scale is read once per two rows
    dim3 g2((unsigned)((n_rows + 1) / 2));
#define ATTR_R2(CH)                                                                        \
  hipLaunchKernelGGL((rowscale2_kernel<TX, TY, CH>), g2, block, 0, s, x, ldx, n_rows, D, m, \
                     unit, row_ss, n_ss, y, ldy)
    if (n8 <= 256) ATTR_R2(1);
    else if (n8 <= 512) ATTR_R2(2);
    else ATTR_R2(4);
#undef ATTR_R2
    return hipGetLastError();
  }
  if (n8 <= 256) ATTR_RS(1);
  else if (n8 <= 512) ATTR_RS(2);
  else if (n8 <= 1024) ATTR_RS(4);
  else if (n8 <= 2048) ATTR_RS(8);
  else if (n8 <= 4096) ATTR_RS(16);
  else ATTR_RS(0);
#undef ATTR_RS
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// colsumsq
// ---------------------------------------------------------------------------
constexpr int kColBlock = 256 * 8;  // columns per workgroup

template <typename TX>
__global__ __launch_bounds__(256) void colsumsq_kernel(const TX* __restrict__ X, int64_t ldx,
                                                       int64_t n_rows, int64_t D,
                                                       int64_t rows_per_panel,
                                                       double* __restrict__ part) {
  const int64_t c0 = (int64_t)blockIdx.x * kColBlock + (int64_t)threadIdx.x * 8;
  const int64_t panel = blockIdx.y;
  if (c0 >= D) return;
  const int64_t r0 = panel * rows_per_panel;
  int64_t r1 = r0 + rows_per_panel;
  r1 = r1 > n_rows ? n_rows : r1;
  double acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.0;
  int64_t r = r0;
  for (; r + 8 <= r1; r += 8) {
    float v[8][8];
#pragma unroll
    for (int u = 0; u < 8; ++u) load8_nt<TX>(X + (r + u) * ldx + c0, v[u]);
    float f[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      f[e] = 0.f;
#pragma unroll
      for (int u = 0; u < 8; ++u) f[e] += v[u][e] * v[u][e];
      acc[e] += (double)f[e];
    }
  }
  for (; r < r1; ++r) {
    float v[8];
    load8<TX>(X + r * ldx + c0, v);
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] += (double)(v[e] * v[e]);
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) part[panel * D + c0 + e] = acc[e];
}

// h_j += sum over panels of part[p][j]: a workgroup takes 64 columns, wave w
// sums panels p = w (mod 4) in increasing order (each panel read as 512
// contiguous bytes per wave), and the four sums are added in wave order:
// a fixed order, so the result is deterministic.
__global__ __launch_bounds__(256) void colsumsq_final_kernel(const double* __restrict__ part,
                                                             int64_t n_panels, int64_t D,
                                                             float* __restrict__ H) {
  __shared__ double red[4][64];
  const int w = threadIdx.x >> 6, c = threadIdx.x & 63;
  const int64_t j = (int64_t)blockIdx.x * 64 + c;
  double s = 0.0;
  if (j < D) {
    int64_t p = w;
    for (; p + 12 < n_panels; p += 16) {
      const double v0 = part[p * D + j], v1 = part[(p + 4) * D + j];
      const double v2 = part[(p + 8) * D + j], v3 = part[(p + 12) * D + j];
      s += v0;
      s += v1;
      s += v2;
      s += v3;
    }
    for (; p < n_panels; p += 4) s += part[p * D + j];
  }
  red[w][c] = s;
  __syncthreads();
  if (w == 0 && j < D) H[j] = (float)((double)H[j] + (((red[0][c] + red[1][c]) + red[2][c]) + red[3][c]));
}

}  // namespace

hipError_t launch_rowscale(int x_dtype, int y_dtype, const void* X, int64_t ldx,
                           int64_t n_rows, int64_t D, const float* m, int unit,
                           const float* row_ss, const int8_t* seg_e, int64_t n_ss, void* Y,
                           int64_t ldy, hipStream_t s) {
  if (x_dtype == 0 && y_dtype == 0)
    return launch_rowscale_t<float, float>(X, ldx, n_rows, D, m, unit, row_ss, seg_e, n_ss, Y, ldy, s);
  if (x_dtype == 0 && y_dtype == 2)
    return launch_rowscale_t<float, _Float16>(X, ldx, n_rows, D, m, unit, row_ss, seg_e, n_ss, Y, ldy,
                                              s);
  if (x_dtype == 2 && y_dtype == 0)
    return launch_rowscale_t<_Float16, float>(X, ldx, n_rows, D, m, unit, row_ss, seg_e, n_ss, Y, ldy,
                                              s);
  return launch_rowscale_t<_Float16, _Float16>(X, ldx, n_rows, D, m, unit, row_ss, seg_e, n_ss, Y,
                                               ldy, s);
}

int colsumsq_panels(int64_t n_rows, int64_t D) {
  const int64_t ncb = (D + kColBlock - 1) / kColBlock;
  int64_t panels = (2048 + ncb - 1) / ncb;
  const int64_t max_by_rows = (n_rows + 63) / 64;  // at least 64 rows per panel
  if (panels > max_by_rows) panels = max_by_rows;
  if (panels < 1) panels = 1;
  if (panels > 65535) panels = 65535;
  return (int)panels;
}

hipError_t launch_colsumsq(int x_dtype, const void* X, int64_t ldx, int64_t n_rows, int64_t D,
                           float* H, double* part, hipStream_t s) {
  const int panels = colsumsq_panels(n_rows, D);
  const int64_t rpp = (n_rows + panels - 1) / panels;
  dim3 grid((unsigned)((D + kColBlock - 1) / kColBlock), (unsigned)panels), block(256);
  if (x_dtype == 0)
    hipLaunchKernelGGL(colsumsq_kernel<float>, grid, block, 0, s, (const float*)X, ldx, n_rows, D, rpp, part);
  else if (x_dtype == 1)
    hipLaunchKernelGGL(colsumsq_kernel<__bf16>, grid, block, 0, s, (const __bf16*)X, ldx, n_rows, D, rpp, part);
  else
    hipLaunchKernelGGL(colsumsq_kernel<_Float16>, grid, block, 0, s, (const _Float16*)X, ldx, n_rows, D, rpp, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  dim3 g2((unsigned)((D + 63) / 64));
  hipLaunchKernelGGL(colsumsq_final_kernel, g2, block, 0, s, (const double*)part, (int64_t)panels, D, H);
  return hipGetLastError();
}

}  // namespace attr
