// Device-side helpers shared by the gfx950 kernels of libwide.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace wide {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

// bf16 bit pattern -> fp32 (exact).
__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(((uint32_t)b) << 16);
}

// fp32 -> bf16 bit pattern, round to nearest even; NaN stays a quiet NaN.
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x0040u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return (uint32_t)f32_to_bf16(lo) | ((uint32_t)f32_to_bf16(hi) << 16);
}

// The same rounding (to nearest even) in one v_cvt_pk_bf16_f32.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2_hw(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){lo, hi}, bf16x2_t));
}

// One value through the same instruction (finite values round exactly as
// f32_to_bf16 does).
__device__ __forceinline__ uint16_t f32_to_bf16_hw(float f) { return (uint16_t)pack_bf16x2_hw(f, 0.0f); }

// SiLU in fp32: a * 1/(1 + e^-a) with the hardware reciprocal (about 1 ulp),
// rather than an IEEE division (a dozen instructions per output).
__device__ __forceinline__ float silu(float a) { return a * __builtin_amdgcn_rcpf(1.0f + __expf(-a)); }

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) {
  return __builtin_bit_cast(bf16x8, v);
}

// 32x32x16 bf16 MFMA, fp32 accumulate.  Operand fragments: lane l holds
// A[row = l%32][k = (l/32)*8 .. +8] and B[col = l%32][k = (l/32)*8 .. +8].
// Result: lane l, element i holds C[row = (i/4)*8 + (l/32)*4 + i%4][col = l%32].
__device__ __forceinline__ f32x16 mfma32(u32x4 a, u32x4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a), as_bf16x8(b), c, 0, 0, 0);
}

// 16x16x32 bf16 MFMA.  Lane l holds A[row = l%16][k = (l/16)*8 .. +8] and
// B[col = l%16][k = (l/16)*8 .. +8]; result element i is
// C[row = (l/16)*4 + i][col = l%16].
__device__ __forceinline__ f32x4 mfma16(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a), as_bf16x8(b), c, 0, 0, 0);
}

__device__ __forceinline__ u32x4 ldg16(const void* p) {
  return *reinterpret_cast<const u32x4*>(p);
}

__device__ __forceinline__ void stg16(void* p, u32x4 v) {
  *reinterpret_cast<u32x4*>(p) = v;
}

// Predicated 16-byte loads without branches: a raw buffer view of
// [base, base + bytes) (bytes < 2^31).  A lane whose byte offset lies at or
// past the end (kOffNone) reads zeros and touches no memory -- the buffer
// unit's range check -- so lanes that must contribute nothing need neither a
// branch nor a select around the load.
typedef __amdgpu_buffer_rsrc_t bufview_t;
constexpr uint32_t kOffNone = 0xFFFFFFF0u;

// A pointer the whole wave shares, moved to scalar registers: a buffer view
// built from a value the compiler cannot prove uniform is loaded through a
// per-lane loop over the distinct values.
template <class T>
__device__ __forceinline__ T* uniform_ptr(T* p) {
  const uint64_t v = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return reinterpret_cast<T*>(((uint64_t)hi << 32) | lo);
}

__device__ __forceinline__ bufview_t buf_view(const void* base, uint32_t bytes) {
  // third descriptor word of the gfx9 family: 32-bit data format, no swizzle
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

__device__ __forceinline__ u32x4 buf_ld16(bufview_t v, uint32_t byte_off) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(v, (int)byte_off, 0, 0));
}

// The same with a workgroup-uniform part of the offset in a scalar register.
// The range check applies to the sum (dword by dword): a lane reads zeros
// where byte_off + uniform_off lies past the view's end.
__device__ __forceinline__ u32x4 buf_ld16s(bufview_t v, uint32_t byte_off, uint32_t uniform_off) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(v, (int)byte_off, (int)uniform_off, 0));
}

__device__ __forceinline__ uint16_t buf_ld2(bufview_t v, uint32_t byte_off) {
  return __builtin_bit_cast(uint16_t, __builtin_amdgcn_raw_buffer_load_b16(v, (int)byte_off, 0, 0));
}

// wave index inside the workgroup, as a wave-uniform (scalar) value
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x / kWave); }
__device__ __forceinline__ int lane_id() { return threadIdx.x % kWave; }

}  // namespace wide
