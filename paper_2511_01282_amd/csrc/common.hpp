// Device helpers shared by the verification kernels (gfx950 / CDNA4).
//
// Matrix-core fragments.  Every MFMA operand used here is described by the
// same unit: each lane of a wave holds 16 contiguous bytes of one matrix row,
// lane l covering row (l % 16) and the (l / 16)-th 16-byte piece of a 64-byte
// K-chunk.  mma_k64() contracts one such K-chunk:
//   bf16:  one v_mfma_f32_16x16x32_bf16  (8 elements per lane)
//   f32:   four v_mfma_f32_16x16x4_f32   (4 elements per lane, one per MFMA)
// A and B use the same piece-to-K assignment, so the contraction is exact
// whatever order the hardware consumes the K index in.
// Output: lane l holds C[4 * (l / 16) + i][l % 16], i = 0..3.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace respec {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

struct bf16_t {
  uint16_t bits;
};

constexpr float kNegInf = -__builtin_huge_valf();

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// float32 -> bf16, round to nearest even; NaN stays a quiet NaN.
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7F800000u) == 0x7F800000u) return (uint16_t)((u | ((u & 0x7FFFFFu) ? 0x400000u : 0u)) >> 16);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

template <typename T>
struct Elem;
template <>
struct Elem<bf16_t> {
  static constexpr int kBytes = 2;
  __device__ static float to_f32(const void* base, size_t i) { return bf16_to_f32(((const uint16_t*)base)[i]); }
  __device__ static void store(void* base, size_t i, float v) { ((uint16_t*)base)[i] = f32_to_bf16(v); }
};
template <>
struct Elem<float> {
  static constexpr int kBytes = 4;
  __device__ static float to_f32(const void* base, size_t i) { return ((const float*)base)[i]; }
  __device__ static void store(void* base, size_t i, float v) { ((float*)base)[i] = v; }
};

// 16-byte global load (the address must be 16-byte aligned).
__device__ __forceinline__ u32x4 ld16(const void* p) { return *(const u32x4*)p; }

__device__ __forceinline__ f32x4 mma_k64(bf16_t, u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b),
                                                 c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mma_k64(float, u32x4 a, u32x4 b, f32x4 c) {
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
  return c;
}

__device__ __forceinline__ float wave_max(float v) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Ordering of (value, id) candidates: larger value first, then smaller id.
__device__ __forceinline__ bool better(float va, int ia, float vb, int ib) {
  return va > vb || (va == vb && ia < ib);
}

// Intra-wave ordering point for LDS data written and read by the same wave.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

}  // namespace respec
