// Shared device helpers for the gfx950 (CDNA4) kernels: vector types, MFMA
// fragment wrappers, range-checked buffer loads and wave reductions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace attr {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
typedef int32_t i32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

// Raw (stride 0) buffer resource for the gfx9 family: 32-bit element format,
// range checking against num_records on every lane.
constexpr int kRsrcWord3 = 0x00020000;
// Cache policy bit "nt": data streamed once, do not keep it hot in L2/MALL.
constexpr int kAuxStream = 2;

__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           kRsrcWord3);
}

// 16-byte load through a buffer resource; lanes whose offset is outside the
// resource's range read zeros (no memory access is made for them).
__device__ inline i32x4 load16_stream(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kAuxStream);
}
__device__ inline i32x4 load16_cached(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}

// Raw buffer descriptor words (same layout make_rsrc builds), for inline asm.
__device__ inline i32x4 make_desc(const void* base, uint32_t bytes) {
  const uint64_t a = (uint64_t)(uintptr_t)base;
  return i32x4{(int)(uint32_t)a, (int)(uint32_t)((a >> 32) & 0xffffu), (int)bytes, kRsrcWord3};
}

// The descriptor d moved on by off bytes: base + off and range - off, or
// range 0 (every lane out of range) when live is false or the range is
// empty.  The caller guarantees off < range when live and the range is not
// empty (a live K-stage starts inside the operand's first row).  The GEMM
// cores advance their operand descriptors by one K-stage this way, with
// scalar arithmetic once per stage, so that the per-lane offsets of their
// loads stay fixed (no vector address arithmetic per load) and the range
// check still ends at the operand's last row.  (A clamped subtraction here
// would be selected as a vector instruction.)
__device__ inline i32x4 desc_at(const i32x4& d, uint32_t off, bool live) {
  const uint64_t b = (((uint64_t)(uint32_t)d.y << 32) | (uint32_t)d.x) + off;
  const uint32_t r = (uint32_t)d.z;
  return i32x4{(int)(uint32_t)b, (int)(uint32_t)(b >> 32), (int)(live && r != 0u ? r - off : 0u), d.w};
}

// Direct-to-LDS 16-byte buffer load: lane l's 16 bytes at voff land at LDS
// byte address lds_base + 16 l (lanes out of the descriptor's range write
// zeros).  Issued through inline asm so that the compiler does not add its
// own conservative wait before every later LDS read; the caller owns the
// vmcnt accounting (one instruction per call) and the barrier.
// The descriptor and the LDS base must be wave-uniform; they are passed
// through readfirstlane so that the compiler, when it cannot prove that,
// does not wrap the instruction in a waterfall loop.
__device__ inline i32x4 uniform_desc(const i32x4& d) {
  return i32x4{__builtin_amdgcn_readfirstlane(d.x), __builtin_amdgcn_readfirstlane(d.y),
               __builtin_amdgcn_readfirstlane(d.z), __builtin_amdgcn_readfirstlane(d.w)};
}
__device__ inline void lds_dma16(const i32x4& desc, uint32_t voff, uint32_t lds_base) {
  asm volatile(
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"
      "buffer_load_dwordx4 %0, %1, 0 offen lds"
      :
      : "v"(voff), "s"(uniform_desc(desc)), "s"(__builtin_amdgcn_readfirstlane(lds_base))
      : "memory", "m0");
}
__device__ inline void lds_dma16_nt(const i32x4& desc, uint32_t voff, uint32_t lds_base) {
  asm volatile(
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"
      "buffer_load_dwordx4 %0, %1, 0 offen nt lds"
      :
      : "v"(voff), "s"(uniform_desc(desc)), "s"(__builtin_amdgcn_readfirstlane(lds_base))
      : "memory", "m0");
}

// Direct-to-LDS load with the LDS base already in M0 (set_m0): the
// instruction offset OFF is added to both the memory offset and the LDS
// address, so up to four consecutive 1 KB destinations share one M0 write
// (the caller subtracts OFF from voff).
__device__ inline void set_m0(uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0" : : "s"(__builtin_amdgcn_readfirstlane(lds_base)) : "memory", "m0");
}
template <int OFF>
__device__ inline void lds_dma16_m0(const i32x4& desc, uint32_t voff) {
  static_assert(OFF >= 0 && OFF < 4096, "12-bit instruction offset");
  asm volatile("buffer_load_dwordx4 %0, %1, 0 offen offset:%2 lds"
               :
               : "v"(voff), "s"(uniform_desc(desc)), "n"(OFF)
               : "memory");
}
// The same with the non-temporal cache policy (data read once).
template <int OFF>
__device__ inline void lds_dma16_m0_nt(const i32x4& desc, uint32_t voff) {
  static_assert(OFF >= 0 && OFF < 4096, "12-bit instruction offset");
  asm volatile("buffer_load_dwordx4 %0, %1, 0 offen offset:%2 nt lds"
               :
               : "v"(voff), "s"(uniform_desc(desc)), "n"(OFF)
               : "memory");
}

// s_waitcnt lgkmcnt(0) through the builtin, so that the compiler's own wait
// insertion knows every LDS read before it has completed (an inline-asm wait
// is opaque to it and would be followed by redundant waits); the empty asm
// keeps memory operations from moving across it.
__device__ inline void wait_lgkm0() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);  // vmcnt 63, expcnt 7, lgkmcnt 0
  asm volatile("" ::: "memory");
}

// One 16-byte A fragment times one 16-byte B fragment on the matrix cores,
// accumulated into a 16x16 fp32 tile.  For bf16/fp16 a fragment is 8 values
// of K (one 16x16x32 MFMA); for fp32 it is 4 values of K (four 16x16x4
// MFMAs).  A and B fragments must use the same lane -> K assignment.
struct Bf16Tag {};
struct F16Tag {};
struct F32Tag {};

__device__ inline f32x4 mma16(Bf16Tag, i32x4 a, i32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}
__device__ inline f32x4 mma16(F16Tag, i32x4 a, i32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a),
                                                __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
}
__device__ inline f32x4 mma16(F32Tag, i32x4 a, i32x4 b, f32x4 c) {
  // Bit-cast whole vectors: a bit-cast of a single vector element is not
  // reliable in this compiler (it reads element 0).
  const f32x4 af = __builtin_bit_cast(f32x4, a);
  const f32x4 bf = __builtin_bit_cast(f32x4, b);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(af.x, bf.x, c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(af.y, bf.y, c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(af.z, bf.z, c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(af.w, bf.w, c, 0, 0, 0);
  return c;
}

__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

__device__ inline double wave_sum(double v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

}  // namespace attr
