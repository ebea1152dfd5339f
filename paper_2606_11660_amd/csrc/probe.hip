// Calibration kernels: the HBM read bandwidth and the fp16 matrix-core rate
// that this GPU actually sustains, measured beside the nominal peaks (8 TB/s,
// 2.5 PFLOP/s dense fp16/bf16) that every roofline fraction is quoted
// against.  Neither is part of the attribution method.
#include "common.h"
#include "kernels.h"

namespace attr {
namespace {

// Streaming read of `n16` 16-byte vectors: each workgroup reads 32 KB
// contiguous pieces (eight non-temporal 16-byte loads per thread, each
// guarded by the bound) in a grid-stride loop and folds them into a
// register; the result is stored only if it equals an improbable pattern, so
// the loads stay live without a write stream.
__global__ __launch_bounds__(256) void probe_read_kernel(const i32x4* __restrict__ x, int64_t n16,
                                                         uint32_t* __restrict__ sink) {
  constexpr int U = 8;
  const int64_t stride = (int64_t)gridDim.x * 256 * U;
  i32x4 acc = i32x4{0, 0, 0, 0};
  for (int64_t i = (int64_t)blockIdx.x * 256 * U + threadIdx.x; i < n16; i += stride) {
    i32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u)
      v[u] = i + u * 256 < n16 ? __builtin_nontemporal_load(x + i + u * 256) : i32x4{0, 0, 0, 0};
#pragma unroll
    for (int u = 0; u < U; ++u) acc ^= v[u];
  }
  const uint32_t h = (uint32_t)(acc.x ^ acc.y ^ acc.z ^ acc.w);
  if (h == 0x9e3779b9u) sink[0] = h;
}

// n_mfma 16x16x32 fp16 MFMAs per wave in eight independent accumulator
// chains, operands in registers (no memory traffic).
__global__ __launch_bounds__(256, 2) void probe_mfma_kernel(int64_t n_mfma, float* __restrict__ sink) {
  const int lane = threadIdx.x & 63;
  // fp16 pairs in [0.5, 1): normal values, so no input is a subnormal
  const i32x4 a = (i32x4{lane, lane + 1, lane + 2, lane + 3} & 0x03ff03ff) | 0x38003800;
  const i32x4 b = (i32x4{lane + 5, lane + 6, lane + 7, lane + 8} & 0x03ff03ff) | 0x38003800;
  f32x4 acc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int64_t it = 0; it < n_mfma; it += 8) {
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = mma16(F16Tag{}, a, b, acc[j]);
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j) s += acc[j].x + acc[j].y + acc[j].z + acc[j].w;
  if (s == 1234.5f) sink[0] = s;
}

}  // namespace

hipError_t launch_probe_read(const void* x, size_t bytes, void* sink, hipStream_t s) {
  const int64_t n16 = (int64_t)(bytes / 16);
  hipLaunchKernelGGL(probe_read_kernel, dim3(8192), dim3(256), 0, s, (const i32x4*)x, n16,
                     (uint32_t*)sink);
  return hipGetLastError();
}

hipError_t launch_probe_mfma(int64_t n_mfma, void* sink, hipStream_t s) {
  // two workgroups of four waves per CU: two waves per SIMD on 256 CUs
  hipLaunchKernelGGL(probe_mfma_kernel, dim3(512), dim3(256), 0, s, n_mfma, (float*)sink);
  return hipGetLastError();
}

}  // namespace attr
