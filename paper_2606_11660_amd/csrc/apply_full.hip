// Full second-moment preconditioner applied to store rows: y = M x for every
// row x, with M = (G^T G / N)^{-1/2} (the flat autocorrelation / empirical
// Fisher preconditioner of the method-family table), followed by unit
// normalisation (section "Attribution Pipelines").
//
// M arrives in fp32.  Preparatory kernels find max|M| and split the scaled
// matrix A = 2^s M (s chosen so that max|A| <= 2^15) into two fp16 matrices
// on the same scale, A_hi = fp16(A) and A_lo = fp16(A - A_hi), so that
// A_hi + A_lo equals A to about 22 significant bits: the preconditioner is
// badly conditioned and an fp16 (or bf16) M alone perturbs the whitened
// rows by percents.  Y = 2^-s X (A_hi + A_lo)^T is then one MFMA GEMM whose
// K loop takes each 64-wide block of X against A_hi and then A_lo into the
// same fp32 accumulators (X is read once);
// the epilogue applies 2^-s, writes Y and per-row partial sums of squares
// (from the fp32 values), which the row-scale kernel turns into the
// unit-norm scale in a second pass.  With unit normalisation into an fp16
// Y, each (row, 128-column segment) is written as y 2^-e with e chosen so
// that the segment's largest magnitude lands in [2^13, 2^14): the
// un-normalised rows of a whitened store are not bounded (H^{-1/2}
// amplifies the directions of the smallest kept eigenvalues by up to
// ~10^4), so y itself may exceed fp16's range, while the unit row never
// does.  e goes to the workspace beside the partial sums and the second
// pass multiplies it back into the row scale; for rows within fp16's normal
// range the results are the same bits as an unscaled intermediate.
#include "common.h"
#include "gemm.h"
#include "kernels.h"

namespace attr {
namespace {

// max|M| as the bit pattern of a non-negative float (integer order equals
// float order there), so the reduction is exact and order independent.
__global__ __launch_bounds__(256) void absmax_kernel(const float* __restrict__ M, int64_t n,
                                                     unsigned int* __restrict__ out) {
  float m = 0.f;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    m = fmaxf(m, fabsf(M[i]));
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) m = fmaxf(m, __shfl_xor(m, off, kWave));
  if ((threadIdx.x & 63) == 0) atomicMax(out, __float_as_uint(m));
}

__global__ void zero_word_kernel(unsigned int* p) { *p = 0u; }

// exponent s with max|M| * 2^s <= 2^15 (0 for an all-zero M)
__device__ inline int split_exponent(unsigned int maxbits) {
  const float mx = __uint_as_float(maxbits);
  if (!(mx > 0.f)) return 0;
  int e;
  frexpf(mx, &e);  // mx = f * 2^e, f in [0.5, 1)
  return 15 - e;
}

__global__ __launch_bounds__(256) void split_m_kernel(const float* __restrict__ M, int64_t n,
                                                      const unsigned int* __restrict__ maxbits,
                                                      _Float16* __restrict__ hi,
                                                      _Float16* __restrict__ lo) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  const float a = ldexpf(M[i], split_exponent(*maxbits));
  const _Float16 h = (_Float16)a;
  hi[i] = h;
  lo[i] = (_Float16)(a - (float)h);
}

template <typename YT>
__device__ inline void store_y(YT* p, float v);
template <>
__device__ inline void store_y<float>(float* p, float v) {
  *p = v;
}
template <>
__device__ inline void store_y<_Float16>(_Float16* p, float v) {
  *p = (_Float16)v;
}

template <typename YT>
__global__ __launch_bounds__(256) void apply_full_kernel(
    const _Float16* __restrict__ X, int64_t n_rows, int64_t ldx, int64_t D,
    const _Float16* __restrict__ Mhi, const _Float16* __restrict__ Mlo,
    const unsigned int* __restrict__ maxbits, YT* __restrict__ Y, int64_t ldy,
    float* __restrict__ rowss, int8_t* __restrict__ rowexp, int n_ss, int n_tn) {
  __shared__ GemmSmem sm;
  const int tn = (int)(blockIdx.x % (uint32_t)n_tn);
  const int64_t tm = blockIdx.x / (uint32_t)n_tn;
  const int64_t r0 = tm * GT, c0 = (int64_t)tn * GT;
  int64_t nr = n_rows - r0;
  nr = nr > GT ? GT : nr;
  int64_t nc = D - c0;
  nc = nc > GT ? GT : nc;
  const i32x4 dx = make_desc(X + r0 * ldx, (uint32_t)(nr * ldx * 2));
  const i32x4 dlo = make_desc(Mlo + c0 * D, (uint32_t)(nc * D * 2));
  const i32x4 dhi = make_desc(Mhi + c0 * D, (uint32_t)(nc * D * 2));
  GemmCoreHL<F16Tag> core;
  core.zero();
  core.run(sm, dx, ldx, dhi, dlo, D, (int)(D / GKS));
  const float unscale = ldexpf(1.f, -split_exponent(*maxbits));

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = GemmCore<F16Tag>::row_of(i, r);  // same layout as GemmCoreHL
      float v[8];
      float ss = 0.f, mx = 0.f;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int col = GemmCore<F16Tag>::col_of(j);
        v[j] = row < nr && col < nc ? core.acc[i][j][r] * unscale : 0.f;
        ss += v[j] * v[j];
        mx = fmaxf(mx, fabsf(v[j]));
      }
      // reduce over the 16 lanes that share this row (128 columns)
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) {
        ss += __shfl_xor(ss, o, kWave);
        mx = fmaxf(mx, __shfl_xor(mx, o, kWave));
      }
      int e = 0;
      if (rowexp && mx > 0.f && mx <= 3.4e38f) {
        int ex;
        frexpf(mx, &ex);  // mx = f 2^ex, f in [0.5, 1)
        e = ex - 14;
        e = e < -120 ? -120 : (e > 120 ? 120 : e);
      }
      const float down = ldexpf(1.f, -e);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int col = GemmCore<F16Tag>::col_of(j);
        if (row < nr && col < nc) store_y<YT>(Y + (r0 + row) * ldy + c0 + col, v[j] * down);
      }
      if (rowss && (lane & 15) == 0 && row < nr) {
        const int64_t at = (r0 + row) * n_ss + 2 * tn + (wave & 1);
        rowss[at] = ss;
        if (rowexp) rowexp[at] = (int8_t)e;
      }
    }
}

}  // namespace

int apply_full_nss(int64_t D) { return (int)(2 * ((D + GT - 1) / GT)); }

hipError_t launch_apply_full(const void* X, int64_t n_rows, int64_t ldx, int64_t D, const float* M,
                             int y_dtype, void* Y, int64_t ldy, int unit, void* ws,
                             hipStream_t s) {
  char* base = static_cast<char*>(ws);
  const size_t mbytes = (size_t)D * (size_t)D * 2;
  const size_t mb_al = (mbytes + 255) / 256 * 256;
  _Float16* hi = reinterpret_cast<_Float16*>(base);
  _Float16* lo = reinterpret_cast<_Float16*>(base + mb_al);
  unsigned int* maxbits = reinterpret_cast<unsigned int*>(base + 2 * mb_al);
  const int n_ss = apply_full_nss(D);
  const size_t ss_bytes = ((size_t)n_rows * (size_t)n_ss * 4 + 255) / 256 * 256;
  float* rowss = unit ? reinterpret_cast<float*>(base + 2 * mb_al + 256) : nullptr;
  // segment exponents only where the un-normalised rows pass through fp16
  int8_t* rowexp = unit && y_dtype == 2
                       ? reinterpret_cast<int8_t*>(base + 2 * mb_al + 256 + ss_bytes)
                       : nullptr;
  const int64_t nm = D * D;
  hipLaunchKernelGGL(zero_word_kernel, dim3(1), dim3(1), 0, s, maxbits);
  hipLaunchKernelGGL(absmax_kernel, dim3(1024), dim3(256), 0, s, M, nm, maxbits);
  hipLaunchKernelGGL(split_m_kernel, dim3((unsigned)((nm + 255) / 256)), dim3(256), 0, s, M, nm,
                     (const unsigned int*)maxbits, hi, lo);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int n_tn = (int)((D + GT - 1) / GT);
  const int64_t n_tm = (n_rows + GT - 1) / GT;
  dim3 grid((unsigned)(n_tm * n_tn)), block(256);
  if (y_dtype == 2)
    hipLaunchKernelGGL(apply_full_kernel<_Float16>, grid, block, 0, s, (const _Float16*)X, n_rows,
                       ldx, D, hi, lo, (const unsigned int*)maxbits, (_Float16*)Y, ldy, rowss, rowexp,
                       n_ss, n_tn);
  else
    hipLaunchKernelGGL(apply_full_kernel<float>, grid, block, 0, s, (const _Float16*)X, n_rows, ldx,
                       D, hi, lo, (const unsigned int*)maxbits, (float*)Y, ldy, rowss, nullptr, n_ss,
                       n_tn);
  e = hipGetLastError();
  if (e != hipSuccess || !unit) return e;
  return launch_rowscale(y_dtype, y_dtype, Y, ldy, n_rows, D, nullptr, 1, rowss, rowexp, n_ss, Y,
                         ldy, s);
}

size_t apply_full_workspace(int64_t n_rows, int64_t D, int unit) {
  const size_t mbytes = (size_t)D * (size_t)D * 2;
  const size_t mb_al = (mbytes + 255) / 256 * 256;
  size_t total = 2 * mb_al + 256;
  // per (row, 128-column segment): fp32 partial sum of squares and the
  // int8 exponent of the fp16 intermediate (the latter only for fp16 Y,
  // but the query has no dtype, so it is always counted)
  if (unit) {
    total += ((size_t)n_rows * (size_t)apply_full_nss(D) * 4 + 255) / 256 * 256;
    total += ((size_t)n_rows * (size_t)apply_full_nss(D) + 255) / 256 * 256;
  }
  return total;
}

}  // namespace attr
